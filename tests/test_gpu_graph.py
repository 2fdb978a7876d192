"""The block forward + backward captured as a HIP graph (how the benchmark
replays a step): every replay must give the eager result bit for bit, also
with other eager work and synchronizations between the replays.

Only the workspace path is captured.  Capturing the direct path crashed
once inside hipStreamEndCapture (a host segmentation fault in the runtime,
at a time when that path ran GEMMs on two streams; the cause was never
identified).  The library refuses a capturing stream whenever a call would
take the direct path (no workspace, one smaller than the pass needs, or a
backward with tokens % 8 != 0), before it enqueues anything, and the direct
cases here stay skipped."""
import pytest
import torch

import paper_2301_08658_amd as atp
from helpers import block_mode_code, block_workspace, group_table, make_block_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _block_call(inp, chunks, workspace):
    """Preallocated outputs and a function that runs fwd then bwd (the
    backward consumes the forward's H and pre-activation) on the current
    stream, with side streams made once."""
    T, G, m, mode = inp["T"], inp["G"], inp["m"], block_mode_code(inp["mode"])
    bf = lambda r, c: torch.empty((r, c), dtype=torch.bfloat16, device=DEV)  # noqa: E731
    own = [torch.empty((T, g.n_loc), device=DEV) if g.red_size > 1 else None for g in G]
    tabs = [group_table(own[i], inp["peers"][i], G[i].red_index) if G[i].red_size > 1 else None
            for i in range(4)]
    bown = [torch.empty((T, g.k_loc), device=DEV) if g.bwd_size > 1 else None for g in G]
    btabs = [group_table(bown[i], inp["dx_peers"][i], G[i].bwd_index) if G[i].bwd_size > 1
             else None for i in range(4)]
    out = dict(qkv=bf(T, G[0].n_loc), o=bf(T, G[1].n_loc), h=bf(T, G[2].n_loc),
               pre=bf(T, G[2].n_loc), z=bf(T, G[3].n_loc), dh_pre=bf(T, G[2].n_loc),
               dx_qkv=bf(T, G[0].k_loc), dx_fc1=bf(T, G[2].k_loc), d_attn=bf(T, G[1].k_loc))
    out.update({f"dw{i}": torch.empty((g.k_loc, g.n_loc), device=DEV) for i, g in enumerate(G)})
    out.update({f"db{i}": torch.empty((g.n_loc,), device=DEV) for i, g in enumerate(G)})
    ws = block_workspace(inp) if workspace else None
    ms = torch.cuda.Stream()

    def call():
        cs = torch.cuda.current_stream()
        atp.atp_block_fwd(m, mode, T, inp["h"], chunks, inp["w"], inp["b"], inp["x"], inp["a"],
                          tabs, out["qkv"], out["o"], out["h"], out["pre"], out["z"],
                          workspace=ws, compute_stream=cs, comm_stream=ms)
        atp.atp_block_bwd(m, mode, T, inp["h"], chunks, inp["w"], inp["b"], inp["x"], inp["a"],
                          out["h"], out["pre"], inp["dz"], inp["dqkv"], inp["do"], btabs,
                          out["dh_pre"], out["dx_qkv"], out["dx_fc1"], out["d_attn"],
                          [out[f"dw{i}"] for i in range(4)], [out[f"db{i}"] for i in range(4)],
                          workspace=ws, compute_stream=cs, comm_stream=ms)
    return out, call


@pytest.mark.parametrize("workspace", [
    True,
    pytest.param(False, marks=pytest.mark.skip(
        reason="capturing the direct path crashed in hipStreamEndCapture once (host segfault "
               "in the runtime, cause not identified); the library refuses it"))],
    ids=["workspace", "direct"])
@pytest.mark.parametrize("case", [("col", (2, 4), (1, 2), 512, 1024, 4),
                                  ("col", (8, 1), (3, 0), 256, 2048, 2),
                                  ("row", (4, 2), (2, 1), 384, 1024, 3)],
                         ids=lambda c: f"{c[0]}{c[1][0]}x{c[1][1]}_c{c[5]}")
def test_graph_replay_equals_eager(case, workspace):
    mode, mesh, coord, T, h, chunks = case
    print(f"graph {case} workspace={workspace}", flush=True)
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=31, bwd=True)
    out, call = _block_call(inp, chunks, workspace)
    call()                                   # eager (also grows the event pool)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    other = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=32, bwd=True)
    other_out, other_call = _block_call(other, chunks, workspace)
    for rep in range(3):
        for v in out.values():               # eager fills between replays
            v.fill_(float("nan"))
        other_call()                         # unrelated eager block work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in out.items():
            assert torch.equal(v.view(torch.int16 if v.element_size() == 2 else torch.int32),
                               ref[k].view(torch.int16 if v.element_size() == 2 else torch.int32)), \
                f"replay {rep}: {k}"
    del other_out


@pytest.mark.parametrize("case", ["fwd_undersized", "bwd_undersized", "bwd_ragged_tokens"])
def test_capture_refused_on_direct_path(case):
    """Under capture, a call that would take the direct path returns
    ATP_ERR_UNSUPPORTED before enqueueing anything: a workspace one piece
    short of the pass's need, or a backward whose token count is not a
    multiple of 8 (with a full workspace).  The capture itself holds one fill
    kernel and ends normally; its replay runs that kernel only."""
    print(f"capture refusal {case}", flush=True)
    T = 132 if case == "bwd_ragged_tokens" else 256
    inp = make_block_inputs("col", (2, 2), (1, 0), T, 512, 0.02, seed=33, bwd=True)
    out, _ = _block_call(inp, 2, False)
    m, mode, G = inp["m"], block_mode_code(inp["mode"]), inp["G"]
    full = atp.atp_block_workspace_bytes(m, mode, T, 512, 2)
    bwd = case.startswith("bwd")
    # the pass's need: the least size (in 256-byte pieces) that takes the path
    need = next(n for n in range(full, 0, -256)
                if atp.atp_block_workspace_path(m, mode, T, 512, atp.ATP_W_KN, n - 256,
                                                int(bwd)) == 0)
    size = full if case == "bwd_ragged_tokens" else need - 256
    assert atp.atp_block_workspace_path(m, mode, T, 512, atp.ATP_W_KN, size, int(bwd)) == 0
    ws = torch.empty(size, dtype=torch.uint8, device=DEV)
    bown = [torch.empty((T, g.k_loc), device=DEV) if g.bwd_size > 1 else None for g in G]
    btabs = [group_table(bown[i], inp["dx_peers"][i], G[i].bwd_index) if G[i].bwd_size > 1
             else None for i in range(4)]
    own = [torch.empty((T, g.n_loc), device=DEV) if g.red_size > 1 else None for g in G]
    tabs = [group_table(own[i], inp["peers"][i], G[i].red_index) if G[i].red_size > 1 else None
            for i in range(4)]
    marker = torch.zeros(64, device=DEV)
    ms = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    err = None
    with torch.cuda.graph(g):
        marker.fill_(1.0)
        cs = torch.cuda.current_stream()
        try:
            if bwd:
                atp.atp_block_bwd(m, mode, T, 512, 2, inp["w"], inp["b"], inp["x"], inp["a"],
                                  inp["hs"], inp["pres"], inp["dz"], inp["dqkv"], inp["do"],
                                  btabs, out["dh_pre"], out["dx_qkv"], out["dx_fc1"],
                                  out["d_attn"], [out[f"dw{i}"] for i in range(4)],
                                  [out[f"db{i}"] for i in range(4)], workspace=ws,
                                  compute_stream=cs, comm_stream=ms)
            else:
                atp.atp_block_fwd(m, mode, T, 512, 2, inp["w"], inp["b"], inp["x"], inp["a"],
                                  tabs, out["qkv"], out["o"], out["h"], out["pre"], out["z"],
                                  workspace=ws, compute_stream=cs, comm_stream=ms)
        except atp.AtpError as e:
            err = e
    torch.cuda.synchronize()
    assert err is not None and err.status == atp.ATP_ERR_UNSUPPORTED, err
    assert "workspace path" in str(err)
    g.replay()
    torch.cuda.synchronize()
    assert torch.all(marker == 1.0)


def _attention_block_call(case, seed, workspace):
    """Seeded inputs of one device's attention block (other members' data
    in place), preallocated outputs, and a function running its forward
    then backward on the current stream."""
    import synth_inputs as S
    mode, mesh, coord, h, heads, batch, seq, chunks = case
    bm = block_mode_code(mode)
    m = atp.mesh(*mesh, *coord)
    gq, go = atp.block_geometry(m, bm, h)[:2]
    _, hd, _ = atp.attention_heads(m, bm, h, heads)
    T = batch * seq
    rnd = lambda shape, std, tid, dt=torch.bfloat16: S.randn_device(  # noqa: E731
        shape, std, seed, tid, DEV, dtype=dt)
    x = rnd((T, gq.k_loc), 1.0, 1)
    wts = [rnd((gq.k_loc, gq.n_loc), 0.02, 2), rnd((go.k_loc, go.n_loc), 0.02, 3)]
    bs = [rnd((gq.n_loc,), 0.02, 4), rnd((go.n_loc,), 0.02, 5)]

    def table(size, idx, cols, tid0):
        return None if size == 1 else [torch.empty((T, cols), device=DEV) if j == idx else
                                       rnd((T, cols), 0.5, tid0 + j, torch.float32)
                                       for j in range(size)]
    qtab, otab = table(gq.red_size, gq.red_index, gq.n_loc, 10), table(go.red_size, go.red_index,
                                                                       go.n_loc, 30)
    atab, xtab = table(go.bwd_size, go.bwd_index, go.k_loc, 50), table(gq.bwd_size, gq.bwd_index,
                                                                       gq.k_loc, 70)
    gathered, dq0, d_o = rnd((T, go.k_loc), 1.0, 6), rnd((T, gq.n_loc), 1.0, 7), rnd((T, go.n_loc),
                                                                                     1.0, 8)
    out = dict(qkv=torch.empty((T, gq.n_loc), dtype=torch.bfloat16, device=DEV),
               attn=gathered.clone(), lse=torch.empty((hd, T), device=DEV),
               o=torch.empty((T, go.n_loc), dtype=torch.bfloat16, device=DEV),
               d_attn=torch.empty((T, go.k_loc), dtype=torch.bfloat16, device=DEV),
               d_qkv=dq0.clone(), dx=torch.empty((T, gq.k_loc), dtype=torch.bfloat16, device=DEV),
               dw0=torch.empty((gq.k_loc, gq.n_loc), device=DEV),
               dw1=torch.empty((go.k_loc, go.n_loc), device=DEV),
               db0=torch.empty((gq.n_loc,), device=DEV), db1=torch.empty((go.n_loc,), device=DEV))
    delta = torch.empty(hd * T, device=DEV)
    ws = None
    if workspace:
        ws = torch.empty(atp.atp_block_workspace_bytes(m, bm, T, h, chunks), dtype=torch.uint8,
                         device=DEV)
    ms = torch.cuda.Stream()

    def call():
        cs = torch.cuda.current_stream()
        # the gathered buffers hold the other members' columns on every call
        out["attn"].copy_(gathered)
        out["d_qkv"].copy_(dq0)
        atp.atp_attention_block_fwd(m, bm, batch, seq, h, heads, chunks, wts, bs, x, qtab,
                                    out["qkv"], out["attn"], out["lse"], otab, out["o"],
                                    workspace=ws, compute_stream=cs, comm_stream=ms)
        atp.atp_attention_block_bwd(m, bm, batch, seq, h, heads, 1, wts, bs, x, out["qkv"],
                                    out["attn"], out["lse"], d_o, atab, out["d_attn"], delta,
                                    out["d_qkv"], xtab, out["dx"], [out["dw0"], out["dw1"]],
                                    [out["db0"], out["db1"]], workspace=ws, compute_stream=cs,
                                    comm_stream=ms)
    return out, call


ATTN_CASES = [("col", (2, 4), (1, 2), 2048, 16, 2, 256, 2),   # forward chunk products split
              ("col", (8, 1), (3, 0), 2048, 16, 1, 512, 4)]


@pytest.mark.parametrize("case", ATTN_CASES, ids=lambda c: f"{c[0]}{c[1][0]}x{c[1][1]}")
def test_attention_block_graph_replay_equals_eager(case):
    """The chained attention block (forward, then backward) on its workspace
    path captured as a HIP graph: three replays, with eager fills and an
    unrelated eager attention block call between them, each give the eager
    result bit for bit."""
    print(f"attention block graph {case}", flush=True)
    out, call = _attention_block_call(case, 35, True)
    call()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    other_out, other_call = _attention_block_call(case, 36, True)
    for rep in range(3):
        for v in out.values():
            v.fill_(float("nan"))
        other_call()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in out.items():
            view = torch.int16 if v.element_size() == 2 else torch.int32
            assert torch.equal(v.view(view), ref[k].view(view)), f"replay {rep}: {k}"
    del other_out


def test_attention_block_capture_refused_without_workspace():
    """Without a workspace the attention block forward returns
    ATP_ERR_UNSUPPORTED on a capturing stream before enqueueing anything; the
    capture (one fill kernel) ends normally."""
    out, _ = _attention_block_call(ATTN_CASES[1], 37, False)
    mode, mesh, coord, h, heads, batch, seq, chunks = ATTN_CASES[1]
    bm = block_mode_code(mode)
    m = atp.mesh(*mesh, *coord)
    gq, go = atp.block_geometry(m, bm, h)[:2]
    T = batch * seq
    x = torch.zeros((T, gq.k_loc), dtype=torch.bfloat16, device=DEV)
    wts = [torch.zeros((gq.k_loc, gq.n_loc), dtype=torch.bfloat16, device=DEV),
           torch.zeros((go.k_loc, go.n_loc), dtype=torch.bfloat16, device=DEV)]
    bs = [torch.zeros(gq.n_loc, dtype=torch.bfloat16, device=DEV),
          torch.zeros(go.n_loc, dtype=torch.bfloat16, device=DEV)]
    otab = [torch.zeros((T, go.n_loc), device=DEV) for _ in range(go.red_size)]
    marker = torch.zeros(64, device=DEV)
    ms = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    err = None
    with torch.cuda.graph(g):
        marker.fill_(1.0)
        try:
            atp.atp_attention_block_fwd(m, bm, batch, seq, h, heads, chunks, wts, bs, x, None,
                                        out["qkv"], out["attn"], out["lse"], otab, out["o"],
                                        compute_stream=torch.cuda.current_stream(),
                                        comm_stream=ms)
        except atp.AtpError as e:
            err = e
    torch.cuda.synchronize()
    assert err is not None and err.status == atp.ATP_ERR_UNSUPPORTED, err
    g.replay()
    torch.cuda.synchronize()
    assert torch.all(marker == 1.0)
