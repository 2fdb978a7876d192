"""Pins of the fp64 oracle against what the paper and mathematics fix.

None of these compare the oracle with itself: the pins are the paper's
worked sharding example (Sec. 3.1), the paper's size formulas (Sec. 3.2),
the special cases of Table 1, brute force over every mesh coordinate
against an independent library product (numpy / torch float64), closed
forms and invariants of GeLU, and torch float64 autograd for the backward
(Sec. 4.2).
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(1234)


def _parse_spec(spec):
    out = []
    for p in spec:
        if p == "Replicate":
            out.append(O.REPLICATE)
        elif p.startswith("Partial"):
            out.append(O.PARTIAL_SUM)
        else:
            out.append(int(p[len("Shard("):-1]))
    return out


# ---------------------------------------------------------------- Sec. 3.1
def test_sharding_example_golden():
    g = json.load(open(os.path.join(GOLDEN, "sharding_example.json")))
    t = np.array(g["tensor"], dtype=np.float64)
    mesh = g["mesh"]
    for case in g["cases"]:
        spec = _parse_spec(case["spec"])
        for rank_s, block in case["rank_blocks"].items():
            coord = O.mesh_coord(mesh, int(rank_s))
            got = O.local_tensor(t, mesh, coord, spec)
            np.testing.assert_array_equal(got, np.array(block, dtype=np.float64))


def test_mesh_rank_row_major_and_roundtrip():
    # Sec. 3.1: [Replicate, Shard(0)] gives ranks 0 and 2 the same block, so
    # ranks 0, 2 share the second mesh coordinate: rank = i1 * d2 + i2.
    assert O.mesh_coord([2, 2], 2) == (1, 0)
    assert O.mesh_coord([2, 2], 1) == (0, 1)
    for mesh in ([2, 2], [2, 4], [4, 2], [8, 1], [1, 8], [3, 5]):
        for r in range(mesh[0] * mesh[1]):
            c = O.mesh_coord(mesh, r)
            assert c == (r // mesh[1], r % mesh[1])
            assert O.mesh_rank(mesh, c) == r


def test_spec_block_rejects_indivisible():
    with pytest.raises(ValueError):
        O.spec_block([2, 2], (0, 0), (0, 1), (3, 4))


# ---------------------------------------------------------------- Table 1
def test_table1_special_cases_1d_mesh():
    T, K, N, d = 6, 8, 12, 4
    X = RNG.standard_normal((T, K))
    W = RNG.standard_normal((K, N))
    ref = X @ W                                   # numpy, not the oracle
    for r in range(d):
        # data parallel: [Shard(0)] x [Replicate] -> [Shard(0)]
        x = O.local_tensor(np.tile(X, (d, 1)), [d], (r,), [0])
        np.testing.assert_allclose(O.matmul(x, W), ref, rtol=1e-13, atol=1e-13)
        # column TP: [Replicate] x [Shard(1)] -> [Shard(1)]
        w = O.local_tensor(W, [d], (r,), [1])
        np.testing.assert_allclose(O.matmul(X, w), ref[:, r * N // d:(r + 1) * N // d],
                                   rtol=1e-13, atol=1e-13)
    # row TP: [Shard(1)] x [Shard(0)] -> [Partial(SUM)]
    parts = [O.matmul(O.local_tensor(X, [d], (r,), [1]), O.local_tensor(W, [d], (r,), [0]))
             for r in range(d)]
    np.testing.assert_allclose(O.partial_reduce(parts)[0], ref, rtol=1e-12, atol=1e-12)


def test_pc_with_d1_1_is_row_tp_and_pr_with_d2_1_is_row_tp():
    # Sec. 3.2.1: DeviceMesh(N, 1) is Megatron's TP.  Row-first with d2 = 1
    # splits W by rows only (Row TP); column-first with d1 = 1 splits W by
    # rows only as well (its first level is trivial), column-first with
    # d2 = 1 splits by columns only (Column TP).
    K, N = 16, 24
    g = O.shard_geometry([4, 1], (2, 0), O.ROW_FIRST, K, N)
    assert (g["k_lo"], g["k_hi"], g["n_lo"], g["n_hi"]) == (8, 12, 0, 24)
    assert (g["red_axis"], g["red_size"], g["red_index"]) == (0, 4, 2)
    g = O.shard_geometry([4, 1], (2, 0), O.COL_FIRST, K, N)
    assert (g["k_lo"], g["k_hi"], g["n_lo"], g["n_hi"]) == (0, 16, 12, 18)
    assert g["red_size"] == 1


# ---------------------------------------------------------------- Sec. 3.2
@pytest.mark.parametrize("mesh", [(2, 2), (2, 4), (4, 2), (8, 1), (1, 8), (3, 2)])
def test_local_sizes_match_paper_formulas(mesh):
    d1, d2 = mesh
    b, h1, h2 = 5, 48, 96
    for i1, i2 in itertools.product(range(d1), range(d2)):
        # row-first: X [b, h1/d1], W [h1/d1, h2/d2], Y [b, h2/d2]
        xs, ws, ys = O.linear_specs(O.ROW_FIRST)
        (xr, xc) = O.spec_block(mesh, (i1, i2), xs, (b, h1))
        (wr, wc) = O.spec_block(mesh, (i1, i2), ws, (h1, h2))
        assert xc[1] - xc[0] == h1 // d1 and xr == (0, b)
        assert (wr[1] - wr[0], wc[1] - wc[0]) == (h1 // d1, h2 // d2)
        g = O.shard_geometry(mesh, (i1, i2), O.ROW_FIRST, h1, h2)
        assert g["n_hi"] - g["n_lo"] == h2 // d2 and g["red_size"] == d1
        # column-first: the communicated tensor is [b, h2/d1]
        g = O.shard_geometry(mesh, (i1, i2), O.COL_FIRST, h1, h2)
        assert g["n_hi"] - g["n_lo"] == h2 // d1 and g["red_size"] == d2
        assert g["k_hi"] - g["k_lo"] == h1 // d2
        # per-rank FMAs b*h1*h2/(d1*d2) for both
        for mode in (O.ROW_FIRST, O.COL_FIRST):
            g = O.shard_geometry(mesh, (i1, i2), mode, h1, h2)
            fma = b * (g["k_hi"] - g["k_lo"]) * (g["n_hi"] - g["n_lo"])
            assert fma * d1 * d2 == b * h1 * h2


@pytest.mark.parametrize("mode", [O.ROW_FIRST, O.COL_FIRST])
@pytest.mark.parametrize("mesh", [(1, 1), (2, 2), (2, 4), (4, 2), (8, 1), (1, 4), (3, 2)])
def test_brute_force_sum_and_concat_equals_unsharded(mesh, mode):
    """Spec invariant: reduce each group's partials, concatenate the
    reduced blocks over the other mesh axis -> the unsharded X W."""
    d1, d2 = mesh
    T, K, N = 7, 24, 48
    X = RNG.standard_normal((T, K))
    W = RNG.standard_normal((K, N))
    ref = X @ W
    got = np.full((T, N), np.nan)
    for i1, i2 in itertools.product(range(d1), range(d2)):
        g = O.shard_geometry(mesh, (i1, i2), mode, K, N)
        group = O.reduction_group(mesh, (i1, i2), g["red_axis"])
        parts = [O.local_partial(X, W, mesh, c, mode) for c in group]
        y, _ = O.partial_reduce(parts)
        np.testing.assert_allclose(y, ref[:, g["n_lo"]:g["n_hi"]], rtol=1e-12, atol=1e-12)
        got[:, g["n_lo"]:g["n_hi"]] = y
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_row_first_equals_column_first_on_transposed_mesh():
    # identity used by the ROW/COL block cross-check: PR(d1,d2;i1,i2) holds
    # the same W block as PC(d2,d1;i2,i1)
    K, N = 24, 48
    for d1, d2 in [(2, 4), (4, 2), (8, 1), (3, 2)]:
        for i1, i2 in itertools.product(range(d1), range(d2)):
            a = O.shard_geometry([d1, d2], (i1, i2), O.ROW_FIRST, K, N)
            b = O.shard_geometry([d2, d1], (i2, i1), O.COL_FIRST, K, N)
            for key in ("k_lo", "k_hi", "n_lo", "n_hi", "red_size", "red_index"):
                assert a[key] == b[key]


# ---------------------------------------------------------------- GEMM
def test_matmul_vs_numpy_and_transposed_views():
    A = RNG.standard_normal((13, 29))
    B = RNG.standard_normal((29, 17))
    np.testing.assert_allclose(O.matmul(A, B), A @ B, rtol=1e-12, atol=1e-12)
    At = np.ascontiguousarray(A.T)
    np.testing.assert_allclose(O.matmul(At.T, B), A @ B, rtol=1e-12, atol=1e-12)
    Bt = np.ascontiguousarray(B.T)
    np.testing.assert_allclose(O.matmul(A, Bt.T), A @ B, rtol=1e-12, atol=1e-12)


def test_matmul_integer_exact():
    A = RNG.integers(-3, 4, (33, 70)).astype(np.float64)
    B = RNG.integers(-3, 4, (70, 41)).astype(np.float64)
    np.testing.assert_array_equal(O.matmul(A, B), (A.astype(np.int64) @ B.astype(np.int64)))


def test_matmul_degenerate_shapes():
    assert O.matmul(np.zeros((0, 4)), np.zeros((4, 3))).shape == (0, 3)
    np.testing.assert_array_equal(O.matmul(np.ones((2, 0)), np.ones((0, 3))), np.zeros((2, 3)))


# ---------------------------------------------------------------- GeLU
def test_gelu_closed_forms_and_torch():
    x = np.concatenate([np.linspace(-8, 8, 401), RNG.standard_normal(200) * 3])
    g = O.gelu(x)
    assert O.gelu(np.array([0.0]))[0] == 0.0
    # GeLU(x) - GeLU(-x) = x  (x*Phi(x) + x*Phi(-x) = x)
    np.testing.assert_allclose(g - O.gelu(-x), x, rtol=0, atol=1e-14)
    # library routine: torch's exact-erf GeLU in float64
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    np.testing.assert_allclose(g, ref, rtol=1e-14, atol=1e-15)
    # tails: GeLU(x) -> x for large x, -> 0 for very negative x
    assert abs(O.gelu(np.array([40.0]))[0] - 40.0) == 0.0
    assert O.gelu(np.array([-40.0]))[0] == 0.0


def test_gelu_grad_vs_autograd_and_finite_difference():
    x = torch.linspace(-6, 6, 241, dtype=torch.float64, requires_grad=True)
    torch.nn.functional.gelu(x, approximate="none").sum().backward()
    got = O.gelu_grad(x.detach().numpy())
    np.testing.assert_allclose(got, x.grad.numpy(), rtol=1e-13, atol=1e-14)
    # central differences of the oracle's own GeLU
    xs = x.detach().numpy()
    eps = 1e-6
    fd = (O.gelu(xs + eps) - O.gelu(xs - eps)) / (2 * eps)
    np.testing.assert_allclose(got, fd, rtol=1e-7, atol=1e-8)
    assert O.gelu_grad(np.array([0.0]))[0] == 0.5


# ---------------------------------------------------------------- bf16 storage
def test_round_bf16_vs_torch_conversion():
    # torch's float32 -> bfloat16 conversion rounds to nearest even; every
    # float32 is exact in float64, so both must agree on float32 inputs
    rng = np.random.default_rng(5)
    x32 = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(3.0),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),       # subnormals
        (rng.standard_normal(2000) * 1e37).astype(np.float32),        # near the top
        np.array([3.3895e38, 3.39e38, -3.4e38, 1e-45, -0.0, 0.0], dtype=np.float32),
    ])
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.round_bf16(x32.astype(np.float64)), ref)


def test_round_bf16_ties_and_specials():
    r = O.round_bf16(np.array([1 + 2**-8, 1 + 3 * 2**-8, -(1 + 2**-8), 1 + 2**-8 + 2**-30,
                               2.0**-133 / 2, 3 * 2.0**-134, np.inf, -np.inf]))
    np.testing.assert_array_equal(r, [1.0, 1 + 2**-6, -1.0, 1 + 2**-7, 0.0, 2 * 2.0**-133,
                                      np.inf, -np.inf])
    assert np.isnan(O.round_bf16(np.array([np.nan]))[0])
    # every bfloat16 value is a fixed point
    allb = torch.arange(0, 2**16, dtype=torch.int32).to(torch.int16).view(torch.bfloat16)
    v = allb.to(torch.float64).numpy()
    v = v[np.isfinite(v)]
    np.testing.assert_array_equal(O.round_bf16(v), v)


# ---------------------------------------------------------------- reduction
def test_partial_reduce_closed_forms():
    T, N = 9, 16
    for d in (1, 2, 3, 8):
        ones = [np.ones((T, N)) for _ in range(d)]
        out, _ = O.partial_reduce(ones)
        np.testing.assert_array_equal(out, np.full((T, N), float(d)))
    ints = [RNG.integers(-1000, 1000, (T, N)).astype(np.float64) for _ in range(5)]
    np.testing.assert_array_equal(O.partial_reduce(ints)[0], np.sum(np.stack(ints), axis=0))
    # d = 1 is a copy
    np.testing.assert_array_equal(O.partial_reduce(ints[:1])[0], ints[0])


def test_partial_reduce_epilogues():
    T, N = 11, 24
    parts = [RNG.standard_normal((T, N)) for _ in range(3)]
    bias = RNG.standard_normal(N)
    s = parts[0] + parts[1] + parts[2]
    out, pre = O.partial_reduce(parts, bias, O.EPI_BIAS)
    np.testing.assert_allclose(out, s + bias, rtol=1e-15, atol=1e-15)
    assert pre is None
    out, pre = O.partial_reduce(parts, bias, O.EPI_BIAS_GELU)
    np.testing.assert_allclose(pre, s + bias, rtol=1e-15, atol=1e-15)
    ref = torch.nn.functional.gelu(torch.from_numpy(s + bias), approximate="none").numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-13, atol=1e-15)
    pin = RNG.standard_normal((T, N))
    out, _ = O.partial_reduce(parts, None, O.EPI_GELU_BWD, pin)
    x = torch.from_numpy(pin).requires_grad_(True)
    torch.nn.functional.gelu(x, approximate="none").backward(torch.from_numpy(s))
    np.testing.assert_allclose(out, x.grad.numpy(), rtol=1e-12, atol=1e-14)


def test_colsum():
    dy = RNG.standard_normal((37, 19))
    np.testing.assert_allclose(O.colsum(dy), dy.sum(axis=0), rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- Sec. 4.2
def test_linear_bwd_vs_autograd():
    T, K, N = 10, 24, 16
    X = torch.randn(T, K, dtype=torch.float64, requires_grad=True)
    W = torch.randn(K, N, dtype=torch.float64, requires_grad=True)
    b = torch.randn(N, dtype=torch.float64, requires_grad=True)
    dY = torch.randn(T, N, dtype=torch.float64)
    (X @ W + b).backward(dY)
    dx, dw, db = O.linear_bwd(X.detach(), W.detach(), dY)
    np.testing.assert_allclose(dx, X.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, W.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, b.grad.numpy(), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- the block
def _global_block(h, T, seed):
    g = torch.Generator().manual_seed(seed)
    shapes = O.block_shapes(h)
    X = torch.randn(T, h, generator=g, dtype=torch.float64)
    A = torch.randn(T, h, generator=g, dtype=torch.float64)
    W = {k: torch.randn(*s, generator=g, dtype=torch.float64) * 0.2 for k, s in shapes.items()}
    B = {k: torch.randn(s[1], generator=g, dtype=torch.float64) * 0.2 for k, s in shapes.items()}
    return X, A, W, B


def _torch_layer(X, A, W, B):
    """Unsharded layer with torch float64 library ops."""
    F = torch.nn.functional
    qkv = F.linear(X, W["qkv"].T, B["qkv"])
    o = F.linear(A, W["out"].T, B["out"])
    pre = F.linear(X, W["fc1"].T, B["fc1"])
    H = F.gelu(pre, approximate="none")
    z = F.linear(H, W["fc2"].T, B["fc2"])
    return dict(qkv=qkv, o=o, pre=pre, h=H, z=z)


def _local_inputs(block_mode, mesh, coord, X, A, W, B):
    """The device's local blocks, cut by the linear specs (Sec. 3.2)."""
    modes = O.block_linear_modes(block_mode)
    w, b = {}, {}
    for name in O.LINEARS:
        xs, ws, ys = O.linear_specs(modes[name])
        w[name] = O.local_tensor(W[name].numpy(), mesh, coord, ws)
        bspec = (ys[0] if ys[0] >= 0 else O.REPLICATE, ys[1] if ys[1] >= 0 else O.REPLICATE)
        # bias follows the output's column split: Shard(1) of Y -> Shard(0) of b
        bspec = tuple(0 if p == 1 else O.REPLICATE for p in bspec)
        b[name] = O.local_tensor(B[name].numpy(), mesh, coord, bspec)
    xs, _, _ = O.linear_specs(modes["qkv"])
    x_loc = O.local_tensor(X.numpy(), mesh, coord, xs)
    xs_o, _, _ = O.linear_specs(modes["out"])
    a_loc = O.local_tensor(A.numpy(), mesh, coord, xs_o)
    return x_loc, a_loc, w, b


@pytest.mark.parametrize("block_mode", [O.BLOCK_COL, O.BLOCK_ROW])
@pytest.mark.parametrize("mesh", [(2, 2), (2, 4), (4, 2), (1, 1)])
def test_block_fwd_global_vs_torch_and_brute_force_local(block_mode, mesh):
    """block_fwd_global against torch (library); block_fwd_local with the true
    partials of every group member against the unsharded layer."""
    h, T = 32, 6
    X, A, W, B = _global_block(h, T, 7)
    ref = _torch_layer(X, A, W, B)
    d1, d2 = mesh
    modes = O.block_linear_modes(block_mode)
    coords = list(itertools.product(range(d1), range(d2)))
    loc = {c: _local_inputs(block_mode, mesh, c, X, A, W, B) for c in coords}
    # first pass: each device's own partials of qkv/out/fc1 and its reduced H
    own = {c: {} for c in coords}
    for c in coords:
        x_loc, a_loc, w, b = loc[c]
        own[c]["qkv"] = O.matmul(x_loc, w["qkv"])
        own[c]["out"] = O.matmul(a_loc, w["out"])
        own[c]["fc1"] = O.matmul(x_loc, w["fc1"])

    def group_peers(c, name, parts_of):
        axis = 1 if modes[name] == O.COL_FIRST else 0
        grp = O.reduction_group(mesh, c, axis)
        return [parts_of(g) for g in grp if g != c]

    H = {}
    for c in coords:
        x_loc, a_loc, w, b = loc[c]
        H[c], _ = O.partial_reduce([own[g]["fc1"] for g in O.reduction_group(
            mesh, c, 1 if modes["fc1"] == O.COL_FIRST else 0)], b["fc1"], O.EPI_BIAS_GELU)
    for c in coords:
        own[c]["fc2"] = O.matmul(H[c], loc[c][2]["fc2"])
    for c in coords:
        x_loc, a_loc, w, b = loc[c]
        peers = {n: group_peers(c, n, lambda g, n=n: own[g][n]) for n in O.LINEARS}
        got = O.block_fwd_local(block_mode, mesh, c, x_loc, a_loc, w, b, peers, round_h=None)
        glob = O.block_fwd_global(block_mode, mesh, c, X, A, W, B)
        for key in ("qkv", "o", "h", "pre", "z"):
            np.testing.assert_allclose(got[key], glob[key], rtol=1e-11, atol=1e-11)
        # global reference vs torch on the same blocks
        for key in ("qkv", "o", "h", "pre", "z"):
            name = dict(qkv="qkv", o="out", h="fc1", pre="fc1", z="fc2")[key]
            _, _, ys = O.linear_specs(modes[name])
            spec = tuple(O.REPLICATE if p == O.PARTIAL_SUM else p for p in ys)
            np.testing.assert_allclose(glob[key], O.local_tensor(ref[key].numpy(), mesh, c, spec),
                                       rtol=1e-12, atol=1e-12)


def test_block_row_on_transposed_mesh_equals_col():
    h, T = 32, 5
    X, A, W, B = _global_block(h, T, 3)
    for (d1, d2) in [(2, 4), (4, 2)]:
        for i1, i2 in itertools.product(range(d1), range(d2)):
            a = O.block_fwd_global(O.BLOCK_COL, (d1, d2), (i1, i2), X, A, W, B)
            b = O.block_fwd_global(O.BLOCK_ROW, (d2, d1), (i2, i1), X, A, W, B)
            for key in a:
                np.testing.assert_array_equal(a[key], b[key])


@pytest.mark.parametrize("block_mode", [O.BLOCK_COL, O.BLOCK_ROW])
@pytest.mark.parametrize("mesh", [(2, 2), (2, 4)])
def test_block_bwd_brute_force_vs_autograd(block_mode, mesh):
    """Every device's reduced input gradients and weight-gradient blocks,
    with true peer partials, against torch float64 autograd of the unsharded
    layer (Sec. 4.2)."""
    h, T = 16, 5
    X, A, W, B = _global_block(h, T, 11)
    Xg = X.clone().requires_grad_(True)
    Ag = A.clone().requires_grad_(True)
    Wg = {k: v.clone().requires_grad_(True) for k, v in W.items()}
    Bg = {k: v.clone().requires_grad_(True) for k, v in B.items()}
    F = torch.nn.functional
    gen = torch.Generator().manual_seed(5)
    dZ = torch.randn(T, h, generator=gen, dtype=torch.float64)
    dQ = torch.randn(T, 3 * h, generator=gen, dtype=torch.float64)
    dO = torch.randn(T, h, generator=gen, dtype=torch.float64)
    # separate leaves for the qkv and fc1 uses of X so the two input
    # gradients can be checked one by one
    Xq = X.clone().requires_grad_(True)
    X1 = X.clone().requires_grad_(True)
    qkv = F.linear(Xq, Wg["qkv"].T, Bg["qkv"])
    o = F.linear(Ag, Wg["out"].T, Bg["out"])
    pre = F.linear(X1, Wg["fc1"].T, Bg["fc1"])
    z = F.linear(F.gelu(pre, approximate="none"), Wg["fc2"].T, Bg["fc2"])
    torch.autograd.backward([z, qkv, o], [dZ, dQ, dO])

    d1, d2 = mesh
    modes = O.block_linear_modes(block_mode)
    coords = list(itertools.product(range(d1), range(d2)))
    fwd = {c: O.block_fwd_global(block_mode, mesh, c, X, A, W, B) for c in coords}
    loc = {c: _local_inputs(block_mode, mesh, c, X, A, W, B) for c in coords}

    def out_block(name, full, c):
        _, _, ys = O.linear_specs(modes[name])
        spec = tuple(O.REPLICATE if p == O.PARTIAL_SUM else p for p in ys)
        return O.local_tensor(full.numpy(), mesh, c, spec)

    grads = {c: dict(fc2=out_block("fc2", dZ, c), qkv=out_block("qkv", dQ, c),
                     out=out_block("out", dO, c)) for c in coords}
    # own dX partials per device and linear (fc1's dY needs the fc2 reduction first)
    own = {c: {} for c in coords}
    for c in coords:
        x_loc, a_loc, w, b = loc[c]
        own[c]["fc2"] = O.matmul(grads[c]["fc2"], w["fc2"].T)
        own[c]["out"] = O.matmul(grads[c]["out"], w["out"].T)
        own[c]["qkv"] = O.matmul(grads[c]["qkv"], w["qkv"].T)

    def bwd_group(c, name):
        axis = 0 if modes[name] == O.COL_FIRST else 1
        return O.reduction_group(mesh, c, axis)

    dpre = {}
    for c in coords:
        dpre[c], _ = O.partial_reduce([own[g]["fc2"] for g in bwd_group(c, "fc2")], None,
                                      O.EPI_GELU_BWD, fwd[c]["pre"])
    for c in coords:
        own[c]["fc1"] = O.matmul(dpre[c], loc[c][2]["fc1"].T)
    for c in coords:
        x_loc, a_loc, w, b = loc[c]
        peers = {n: [own[g][n] for g in bwd_group(c, n) if g != c] for n in O.LINEARS}
        r = O.block_bwd_local(block_mode, mesh, c, x_loc, a_loc, fwd[c]["h"], fwd[c]["pre"], w,
                              grads[c]["fc2"], grads[c]["qkv"], grads[c]["out"], peers,
                              round_dpre=None)
        xs, ws_q, _ = O.linear_specs(modes["qkv"])
        np.testing.assert_allclose(r["dx_qkv"], O.local_tensor(Xq.grad.numpy(), mesh, c, xs),
                                   rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(r["dx_fc1"], O.local_tensor(X1.grad.numpy(), mesh, c, xs),
                                   rtol=1e-11, atol=1e-11)
        xs_o, _, _ = O.linear_specs(modes["out"])
        np.testing.assert_allclose(r["da"], O.local_tensor(Ag.grad.numpy(), mesh, c, xs_o),
                                   rtol=1e-11, atol=1e-11)
        for name in O.LINEARS:
            _, ws, ys = O.linear_specs(modes[name])
            np.testing.assert_allclose(r["dw_" + name],
                                       O.local_tensor(Wg[name].grad.numpy(), mesh, c, ws),
                                       rtol=1e-11, atol=1e-11)
            bspec = tuple(0 if p == 1 else O.REPLICATE for p in ys)
            np.testing.assert_allclose(r["db_" + name],
                                       O.local_tensor(Bg[name].grad.numpy(), mesh, c, bspec),
                                       rtol=1e-11, atol=1e-11)
