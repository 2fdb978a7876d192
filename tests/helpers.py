"""Shared test helpers: tolerance check and device plumbing (no method arithmetic)."""
import numpy as np
import torch

DEV = "cuda:0"

# Tolerance for floating-point parity with the fp64 oracle (bf16 inputs,
# fp32 accumulation, bf16-rounded activations): elementwise
# |gpu - ref| <= 1e-2 * (|ref| + 1) and relative Frobenius error <= 5e-3.
ELEM_TOL = 1e-2
FROB_TOL = 5e-3


def to64(t) -> np.ndarray:
    if isinstance(t, np.ndarray):
        return t.astype(np.float64)
    return t.detach().to("cpu", torch.float64).numpy()


def assert_close(gpu, ref, what="", elem_tol=ELEM_TOL, frob_tol=FROB_TOL, floor=1.0, extra=None):
    """Elementwise |gpu - ref| <= elem_tol * (|ref| + floor) (+ extra, an
    array of per-element error terms derived for a specific computation) and
    relative Frobenius error <= frob_tol.  floor="rms" uses the reference's
    RMS as the absolute floor: for token-sums of a bf16-stored intermediate
    (dW, db of fc1 in the chained backward), where a tie of that intermediate
    rounded the other way moves a whole column by ulp(dY) * |x| whatever the
    column's size."""
    g = to64(gpu)
    r = to64(ref)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite values"
    err = np.abs(g - r)
    if floor == "rms":
        floor = float(np.sqrt(np.mean(r * r))) if r.size else 1.0
    bound = elem_tol * (np.abs(r) + floor)
    if extra is not None:
        bound = bound + to64(extra)
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} elements out of tolerance, first at "
                             f"{tuple(idx)}: gpu={g[tuple(idx)]} ref={r[tuple(idx)]}")
    nr = np.linalg.norm(r)
    if nr > 0:
        rel = np.linalg.norm(g - r) / nr
        assert rel <= frob_tol, f"{what}: relative Frobenius error {rel:.3e} > {frob_tol}"
    return float(err.max()) if err.size else 0.0


def dev(t: torch.Tensor) -> torch.Tensor:
    return t.to(DEV)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to bf16 (RNE) -- used only to build GPU inputs."""
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(
        torch.float64).numpy()


# ---------------------------------------------------------------- block inputs
import paper_2301_08658_amd as atp  # noqa: E402
import synth_inputs as S  # noqa: E402

LIN = ("qkv", "out", "fc1", "fc2")


def block_mode_code(mode: str) -> int:
    return atp.ATP_BLOCK_COL if mode == "col" else atp.ATP_BLOCK_ROW


def make_block_inputs(mode, mesh, coord, T, h, sigma_w, seed, device=DEV, on_device=False,
                      bias_std=0.02, bwd=False, integer=False):
    """Seeded local inputs of one device's block.  Shapes come from the
    library's geometry; values from synth_inputs only.  Peers are the other
    group members' partial buffers (bench mode)."""
    m = atp.mesh(mesh[0], mesh[1], coord[0], coord[1])
    G = atp.block_geometry(m, block_mode_code(mode), h)

    def bf(shape, std, tid):
        if integer:
            return S.randint_bf16(shape, seed, tid).to(device)
        if on_device:
            return S.randn_device(shape, std, seed, tid, device)
        return S.randn_bf16(shape, std, seed, tid).to(device)

    def f32(shape, std, tid):
        if integer:
            return S.randint_f32(shape, seed, tid).to(device)
        if on_device:
            return S.randn_device(shape, std, seed, tid, device, dtype=torch.float32)
        return S.randn_f32(shape, std, seed, tid).to(device)

    inp = dict(m=m, G=G, mode=mode, T=T, h=h)
    inp["x"] = bf((T, G[0].k_loc), 1.0, S.TID["x"])
    inp["a"] = bf((T, G[1].k_loc), 1.0, S.TID["a"])
    inp["w"] = [bf((g.k_loc, g.n_loc), sigma_w, S.TID["w_" + n]) for g, n in zip(G, LIN)]
    inp["b"] = [bf((g.n_loc,), bias_std, S.TID["b_" + n]) if bias_std else
                torch.zeros(g.n_loc, dtype=torch.bfloat16, device=device) for g, n in zip(G, LIN)]
    inp["peers"] = []
    for li, g in enumerate(G):
        sp = S.peer_sigma(g.k_loc, sigma_w, 1.0)
        inp["peers"].append([f32((T, g.n_loc), sp, S.PEER_TID_BASE + 100 * li + j)
                             for j in range(g.red_size - 1)])
    if bwd:
        inp["dz"] = bf((T, G[3].n_loc), 1.0, S.TID["dz"])
        inp["dqkv"] = bf((T, G[0].n_loc), 1.0, S.TID["dqkv"])
        inp["do"] = bf((T, G[1].n_loc), 1.0, S.TID["do"])
        inp["hs"] = bf((T, G[2].n_loc), 0.5, S.TID["h"])
        inp["pres"] = bf((T, G[2].n_loc), 1.0, S.TID["pre"]) if not integer else \
            torch.zeros((T, G[2].n_loc), dtype=torch.bfloat16, device=device)
        inp["dx_peers"] = []
        for li, g in enumerate(G):
            sp = S.peer_sigma(g.n_loc, sigma_w, 1.0)
            inp["dx_peers"].append([f32((T, g.k_loc), sp, S.BWD_PEER_TID_BASE + 100 * li + j)
                                    for j in range(g.bwd_size - 1)])
    return inp


def group_table(own, peers, index):
    """Group-ordered buffer list with the device's own buffer at `index`."""
    return list(peers[:index]) + [own] + list(peers[index:])


def block_workspace(inp):
    """A workspace large enough for the block's transposed-layout path."""
    n = atp.atp_block_workspace_bytes(inp["m"], block_mode_code(inp["mode"]), inp["T"], inp["h"],
                                      1)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=inp["x"].device)


def run_block_fwd(inp, chunks, compute=None, comm=None, same_stream=False, aux=True,
                  workspace=False):
    """Allocate outputs, call atp_block_fwd, return outputs + own partials.
    aux=True also hands the block a second compute stream (accepted and left
    unused by the library); workspace=True
    hands it a workspace, so it runs the transposed-layout path."""
    T, G, m = inp["T"], inp["G"], inp["m"]
    dev_ = inp["x"].device
    own = [torch.full((T, g.n_loc), float("nan"), device=dev_) if g.red_size > 1 else None
           for g in G]
    tabs = [group_table(own[i], inp["peers"][i], G[i].red_index) if G[i].red_size > 1 else None
            for i in range(4)]
    out = dict(qkv=torch.empty((T, G[0].n_loc), dtype=torch.bfloat16, device=dev_),
               o=torch.empty((T, G[1].n_loc), dtype=torch.bfloat16, device=dev_),
               h=torch.empty((T, G[2].n_loc), dtype=torch.bfloat16, device=dev_),
               pre=torch.empty((T, G[2].n_loc), dtype=torch.bfloat16, device=dev_),
               z=torch.empty((T, G[3].n_loc), dtype=torch.bfloat16, device=dev_))
    cs = compute or torch.cuda.current_stream()
    ms = cs if same_stream else (comm or torch.cuda.Stream())
    ax = torch.cuda.Stream() if (aux and not same_stream) else None
    atp.atp_block_fwd(m, block_mode_code(inp["mode"]), T, inp["h"], chunks, inp["w"], inp["b"],
                      inp["x"], inp["a"], tabs, out["qkv"], out["o"], out["h"], out["pre"],
                      out["z"], workspace=block_workspace(inp) if workspace else None,
                      compute_stream=cs, comm_stream=ms, aux_stream=ax)
    out["own"] = own
    return out


def run_block_bwd(inp, chunks, h_act=None, pre=None, same_stream=False, aux=True,
                  workspace=False):
    T, G, m = inp["T"], inp["G"], inp["m"]
    dev_ = inp["x"].device
    h_act = inp["hs"] if h_act is None else h_act
    pre = inp["pres"] if pre is None else pre
    own = [torch.full((T, g.k_loc), float("nan"), device=dev_) if g.bwd_size > 1 else None
           for g in G]
    tabs = [group_table(own[i], inp["dx_peers"][i], G[i].bwd_index) if G[i].bwd_size > 1
            else None for i in range(4)]
    out = dict(dh_pre=torch.empty((T, G[2].n_loc), dtype=torch.bfloat16, device=dev_),
               dx_qkv=torch.empty((T, G[0].k_loc), dtype=torch.bfloat16, device=dev_),
               dx_fc1=torch.empty((T, G[2].k_loc), dtype=torch.bfloat16, device=dev_),
               d_attn=torch.empty((T, G[1].k_loc), dtype=torch.bfloat16, device=dev_),
               dw=[torch.full((g.k_loc, g.n_loc), float("nan"), device=dev_) for g in G],
               db=[torch.full((g.n_loc,), float("nan"), device=dev_) for g in G])
    cs = torch.cuda.current_stream()
    ms = cs if same_stream else torch.cuda.Stream()
    ax = torch.cuda.Stream() if (aux and not same_stream) else None
    atp.atp_block_bwd(m, block_mode_code(inp["mode"]), T, inp["h"], chunks, inp["w"], inp["b"],
                      inp["x"], inp["a"], h_act, pre, inp["dz"], inp["dqkv"], inp["do"], tabs,
                      out["dh_pre"], out["dx_qkv"], out["dx_fc1"], out["d_attn"], out["dw"],
                      out["db"], workspace=block_workspace(inp) if workspace else None,
                      compute_stream=cs, comm_stream=ms, aux_stream=ax)
    out["own"] = own
    return out


def oracle_block_fwd(O, inp, rows=None):
    """Oracle forward of the same device share (bench mode), optionally on a
    subset of token rows (rows are independent in every step)."""
    sel = (lambda t: t) if rows is None else (lambda t: t[rows])
    cpu = lambda t: sel(t.detach().cpu())  # noqa: E731
    bm = O.BLOCK_COL if inp["mode"] == "col" else O.BLOCK_ROW
    w = {n: inp["w"][i].cpu() for i, n in enumerate(LIN)}
    b = {n: inp["b"][i].cpu() for i, n in enumerate(LIN)}
    peers = {n: [cpu(p) for p in inp["peers"][i]] for i, n in enumerate(LIN)}
    return O.block_fwd_local(bm, inp["m"], (inp["m"].i1, inp["m"].i2), cpu(inp["x"]),
                             cpu(inp["a"]), w, b, peers)
