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
