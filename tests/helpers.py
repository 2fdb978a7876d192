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


def assert_close(gpu, ref, what="", elem_tol=ELEM_TOL, frob_tol=FROB_TOL, extra=None):
    """Elementwise |gpu - ref| <= elem_tol * (|ref| + 1) + extra and relative
    Frobenius error <= frob_tol.  `extra` (an array, or a scalar) holds the
    per-element error terms derived for a specific computation from the
    reference's own quantities (tests/bounds.py): the 16-bit handoffs of the
    GPU path that the strict fp64 reference does not make."""
    g = to64(gpu)
    r = to64(ref)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite values"
    err = np.abs(g - r)
    bound = elem_tol * (np.abs(r) + 1.0)
    if extra is not None:
        bound = bound + to64(extra) if not np.isscalar(extra) else bound + float(extra)
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
import bounds  # noqa: E402

LIN = ("qkv", "out", "fc1", "fc2")


def block_mode_code(mode: str) -> int:
    return atp.ATP_BLOCK_COL if mode == "col" else atp.ATP_BLOCK_ROW


def make_block_inputs(mode, mesh, coord, T, h, sigma_w, seed, device=DEV, on_device=False,
                      bias_std=0.02, bwd=False, integer=False, layout=None,
                      partial_dtype=torch.float32):
    """Seeded local inputs of one device's block.  Shapes come from the
    library's geometry; values from synth_inputs only.  Peers are the other
    group members' partial buffers (bench mode), in `partial_dtype`.
    inp["w"] holds the weights as the library receives them (layout
    ATP_W_KN: [k_loc, n_loc]; ATP_W_NK: [n_loc, k_loc] contiguous), inp["wkn"]
    the same values as [k_loc, n_loc] for the oracle."""
    layout = atp.ATP_W_KN if layout is None else layout
    m = atp.mesh(mesh[0], mesh[1], coord[0], coord[1])
    G = atp.block_geometry(m, block_mode_code(mode), h)

    def bf(shape, std, tid):
        if integer:
            return S.randint_bf16(shape, seed, tid).to(device)
        if on_device:
            return S.randn_device(shape, std, seed, tid, device)
        return S.randn_bf16(shape, std, seed, tid).to(device)

    def part(shape, std, tid):
        if integer:
            t = S.randint_f32(shape, seed, tid)
        elif on_device:
            t = S.randn_device(shape, std, seed, tid, device, dtype=torch.float32)
        else:
            t = S.randn_f32(shape, std, seed, tid)
        return t.to(device=device, dtype=partial_dtype)

    inp = dict(m=m, G=G, mode=mode, T=T, h=h, layout=layout, pdt=partial_dtype)
    inp["x"] = bf((T, G[0].k_loc), 1.0, S.TID["x"])
    inp["a"] = bf((T, G[1].k_loc), 1.0, S.TID["a"])
    inp["wkn"] = [bf((g.k_loc, g.n_loc), sigma_w, S.TID["w_" + n]) for g, n in zip(G, LIN)]
    inp["w"] = (inp["wkn"] if layout == atp.ATP_W_KN else
                [w.t().contiguous() for w in inp["wkn"]])
    inp["b"] = [bf((g.n_loc,), bias_std, S.TID["b_" + n]) if bias_std else
                torch.zeros(g.n_loc, dtype=torch.bfloat16, device=device) for g, n in zip(G, LIN)]
    inp["peers"] = []
    for li, g in enumerate(G):
        sp = S.peer_sigma(g.k_loc, sigma_w, 1.0)
        inp["peers"].append([part((T, g.n_loc), sp, S.PEER_TID_BASE + 100 * li + j)
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
            inp["dx_peers"].append([part((T, g.k_loc), sp, S.BWD_PEER_TID_BASE + 100 * li + j)
                                    for j in range(g.bwd_size - 1)])
    return inp


def group_table(own, peers, index):
    """Group-ordered buffer list with the device's own buffer at `index`."""
    return list(peers[:index]) + [own] + list(peers[index:])


def block_workspace(inp):
    """A workspace large enough for the block's transposed-layout path."""
    n = atp.atp_block_workspace_bytes(inp["m"], block_mode_code(inp["mode"]), inp["T"], inp["h"],
                                      1, inp["layout"])
    return torch.empty(max(n, 1), dtype=torch.uint8, device=inp["x"].device)


def nan_like_rows(T, cols, dtype, device):
    """An output buffer poisoned with NaN, so an unwritten element fails."""
    return torch.full((T, cols), float("nan"), dtype=dtype, device=device)


def run_block_fwd(inp, chunks, compute=None, comm=None, same_stream=False, workspace=False):
    """Allocate NaN-poisoned outputs, call atp_block_fwd, return outputs and
    the own partials.  workspace=True hands it a workspace, so it runs the
    transposed-layout path."""
    T, G, m = inp["T"], inp["G"], inp["m"]
    dev_ = inp["x"].device
    pdt = inp["pdt"]
    own = [nan_like_rows(T, g.n_loc, pdt, dev_) if g.red_size > 1 else None for g in G]
    tabs = [group_table(own[i], inp["peers"][i], G[i].red_index) if G[i].red_size > 1 else None
            for i in range(4)]
    bf = torch.bfloat16
    out = dict(qkv=nan_like_rows(T, G[0].n_loc, bf, dev_), o=nan_like_rows(T, G[1].n_loc, bf, dev_),
               h=nan_like_rows(T, G[2].n_loc, bf, dev_), pre=nan_like_rows(T, G[2].n_loc, bf, dev_),
               z=nan_like_rows(T, G[3].n_loc, bf, dev_))
    cs = compute or torch.cuda.current_stream()
    ms = cs if same_stream else (comm or torch.cuda.Stream())
    atp.atp_block_fwd(m, block_mode_code(inp["mode"]), T, inp["h"], chunks, inp["w"], inp["b"],
                      inp["x"], inp["a"], tabs, out["qkv"], out["o"], out["h"], out["pre"],
                      out["z"], workspace=block_workspace(inp) if workspace else None,
                      compute_stream=cs, comm_stream=ms, weight_layout=inp["layout"])
    out["own"] = own
    return out


def run_block_bwd(inp, chunks, h_act=None, pre=None, same_stream=False, workspace=False):
    T, G, m = inp["T"], inp["G"], inp["m"]
    dev_ = inp["x"].device
    h_act = inp["hs"] if h_act is None else h_act
    pre = inp["pres"] if pre is None else pre
    pdt = inp["pdt"]
    own = [nan_like_rows(T, g.k_loc, pdt, dev_) if g.bwd_size > 1 else None for g in G]
    tabs = [group_table(own[i], inp["dx_peers"][i], G[i].bwd_index) if G[i].bwd_size > 1
            else None for i in range(4)]
    bf = torch.bfloat16
    kn = inp["layout"] == atp.ATP_W_KN
    out = dict(dh_pre=nan_like_rows(T, G[2].n_loc, bf, dev_),
               dx_qkv=nan_like_rows(T, G[0].k_loc, bf, dev_),
               dx_fc1=nan_like_rows(T, G[2].k_loc, bf, dev_),
               d_attn=nan_like_rows(T, G[1].k_loc, bf, dev_),
               dw=[torch.full((g.k_loc, g.n_loc) if kn else (g.n_loc, g.k_loc), float("nan"),
                              device=dev_) for g in G],
               db=[torch.full((g.n_loc,), float("nan"), device=dev_) for g in G])
    cs = torch.cuda.current_stream()
    ms = cs if same_stream else torch.cuda.Stream()
    atp.atp_block_bwd(m, block_mode_code(inp["mode"]), T, inp["h"], chunks, inp["w"], inp["b"],
                      inp["x"], inp["a"], h_act, pre, inp["dz"], inp["dqkv"], inp["do"], tabs,
                      out["dh_pre"], out["dx_qkv"], out["dx_fc1"], out["d_attn"], out["dw"],
                      out["db"], workspace=block_workspace(inp) if workspace else None,
                      compute_stream=cs, comm_stream=ms, weight_layout=inp["layout"])
    out["own"] = own
    # dW in the oracle's [k_loc, n_loc] orientation
    out["dw_kn"] = out["dw"] if kn else [d.t() for d in out["dw"]]
    return out


# ---------------------------------------------------------------- oracle side
def _cpu(t):
    return t.detach().cpu()


def oracle_block_fwd(O, inp, rows=None):
    """Strict fp64 oracle forward of the same device share (bench mode),
    optionally on a subset of token rows (rows are independent in every
    step).  Returns the reference dict and the derived per-element terms
    that the GPU's 16-bit handoffs add (bounds module), keyed like it."""
    sel = (lambda t: t) if rows is None else (lambda t: t[rows])
    cpu = lambda t: sel(_cpu(t))  # noqa: E731
    bm = O.BLOCK_COL if inp["mode"] == "col" else O.BLOCK_ROW
    w = {n: _cpu(inp["wkn"][i]) for i, n in enumerate(LIN)}
    b = {n: _cpu(inp["b"][i]) for i, n in enumerate(LIN)}
    peers = {n: [cpu(p) for p in inp["peers"][i]] for i, n in enumerate(LIN)}
    ref = O.block_fwd_local(bm, inp["m"], (inp["m"].i1, inp["m"].i2), cpu(inp["x"]),
                            cpu(inp["a"]), w, b, peers)
    return ref, fwd_extra(O, inp, ref, rows)


def fwd_extra(O, inp, ref, rows=None):
    """Derived terms of the forward: H is handed to fc2 in bf16; with bf16
    partials each reduced output also carries the rounding of the own
    partial (scaled by GeLU' for h, propagated into fc2 through H)."""
    sel = (lambda t: t) if rows is None else (lambda t: t[rows])
    G = inp["G"]
    w = [O._f64(_cpu(t)) for t in inp["wkn"]]
    var_h = bounds.rounding_var(ref["h"])
    extra = {k: 0.0 for k in ("qkv", "o", "h", "pre", "z")}
    if inp["pdt"] == torch.bfloat16:
        ins = [O._f64(sel(_cpu(inp["x"]))), O._f64(sel(_cpu(inp["a"]))),
               O._f64(sel(_cpu(inp["x"])))]
        own = [O.matmul(ins[i], w[i]) if G[i].red_size > 1 else None for i in range(3)]
        if own[0] is not None:
            extra["qkv"] = bounds.single(own[0])
        if own[1] is not None:
            extra["o"] = bounds.single(own[1])
        if own[2] is not None:
            gp = O.gelu_grad(ref["pre"])
            extra["pre"] = bounds.single(own[2])
            extra["h"] = bounds.single(own[2], gp)
            var_h = var_h + (gp * bounds.ulp_bf16(own[2])) ** 2 / 12.0
        if G[3].red_size > 1:
            extra["z"] = bounds.single(O.matmul(ref["h"], w[3]))
    extra["z"] = extra["z"] + bounds.left(var_h, w[3])
    return extra


def oracle_block_bwd(O, inp, round_dpre=None):
    """Strict fp64 oracle backward of the same device share (bench mode) and
    the derived per-element terms of its 16-bit handoffs.  round_dpre (a
    diagnostic mirror, e.g. O.round_bf16) rounds fc1's dY before its backward
    reads it; with it the derived terms are not needed and are zero."""
    bm = O.BLOCK_COL if inp["mode"] == "col" else O.BLOCK_ROW
    coord = (inp["m"].i1, inp["m"].i2)
    w = {n: _cpu(inp["wkn"][i]) for i, n in enumerate(LIN)}
    peers = {n: [_cpu(p) for p in inp["dx_peers"][i]] for i, n in enumerate(LIN)}
    ref = O.block_bwd_local(bm, inp["m"], coord, _cpu(inp["x"]), _cpu(inp["a"]),
                            _cpu(inp["hs"]), _cpu(inp["pres"]), w,
                            _cpu(inp["dz"]), _cpu(inp["dqkv"]), _cpu(inp["do"]), peers,
                            round_dpre=round_dpre)
    if round_dpre is not None:
        return ref, {}
    return ref, bwd_extra(O, inp, ref)


def bwd_extra(O, inp, ref):
    """Derived terms of the backward: dh_pre is handed to fc1's backward in
    bf16 (dX, dW and db of fc1); with bf16 partials each reduced input
    gradient also carries the rounding of the own dX partial."""
    G = inp["G"]
    w = [O._f64(_cpu(t)) for t in inp["wkn"]]
    x = O._f64(_cpu(inp["x"]))
    var_dh = bounds.rounding_var(ref["dh_pre"])
    keys = ("dh_pre", "dx_qkv", "dx_fc1", "da") + tuple(f"{p}_{n}" for p in ("dw", "db")
                                                         for n in LIN)
    extra = {k: 0.0 for k in keys}
    if inp["pdt"] == torch.bfloat16:
        dys = [O._f64(_cpu(inp["dqkv"])), O._f64(_cpu(inp["do"])), ref["dh_pre"],
               O._f64(_cpu(inp["dz"]))]
        own = [O.matmul(dys[i], w[i].T) if G[i].bwd_size > 1 else None for i in range(4)]
        if own[3] is not None:
            gp = O.gelu_grad(O._f64(_cpu(inp["pres"])))
            extra["dh_pre"] = bounds.single(own[3], gp)
            var_dh = var_dh + (gp * bounds.ulp_bf16(own[3])) ** 2 / 12.0
        for i, k in ((0, "dx_qkv"), (1, "da"), (2, "dx_fc1")):
            if own[i] is not None:
                extra[k] = bounds.single(own[i])
    extra["dx_fc1"] = extra["dx_fc1"] + bounds.left(var_dh, w[2].T)
    extra["dw_fc1"] = bounds.right(x, var_dh)
    extra["db_fc1"] = bounds.colsum(var_dh)
    return extra


def check_fwd(out, ref, extra, rows=None, what=""):
    sel = (lambda t: t) if rows is None else (lambda t: t[rows])
    for key in ("qkv", "o", "h", "pre", "z"):
        assert_close(sel(out[key]), ref[key], f"{what} {key}", extra=extra.get(key))


def check_bwd(out, ref, extra, what=""):
    for key in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
        rk = {"d_attn": "da"}.get(key, key)
        assert_close(out[key], ref[rk], f"{what} {key}", extra=extra.get(rk))
    for i, n in enumerate(LIN):
        assert_close(out["dw_kn"][i], ref["dw_" + n], f"{what} dw_{n}", extra=extra.get("dw_" + n))
        assert_close(out["db"][i], ref["db_" + n], f"{what} db_{n}", extra=extra.get("db_" + n))


def assert_paths_agree(a, b, what, rel=1e-4):
    """Two summation orders of the same fp32-accumulated products."""
    if a.dtype == torch.bfloat16:
        # two units in the last place of the larger value (bf16 keeps 8
        # significant bits), plus the fp32 sums' rounding on the tensor's scale
        # for values that come out of cancellation near zero
        fa, fb = a.double(), b.double()
        scale = float(fa.abs().max()) + 1e-30
        bound = 2.0 ** -6 * torch.maximum(fa.abs(), fb.abs()) + rel * scale
        excess = float(((fa - fb).abs() - bound).max())
        assert excess <= 0, f"{what}: bf16 outputs differ beyond two units in the last place"
        frac = float((a.contiguous().view(torch.int16) !=
                      b.contiguous().view(torch.int16)).float().mean())
        assert frac < 0.05, f"{what}: {frac:.3%} of bf16 outputs differ"
    else:
        fa, fb = a.double(), b.double()
        scale = float(fa.abs().max()) + 1e-30
        err = float((fa - fb).abs().max())
        assert err <= rel * scale, f"{what}: max diff {err:.3e} vs scale {scale:.3e}"
