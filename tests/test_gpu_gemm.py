"""GPU parity of the shard-linear GEMMs (Sec. 3.2 forward, Sec. 4.2
backward) against the fp64 oracle.  Integer-valued inputs make every fp32
sum exact, so those cases must match bit for bit; random inputs are held to
the stated tolerance.  Shapes are ragged on purpose (not multiples of the
256 x 256 x 64 tile) and span several tiles."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_08658_amd as atp
import synth_inputs as S
from helpers import DEV, assert_close, to64

pytestmark = pytest.mark.gpu


def _sync():
    torch.cuda.synchronize()


@pytest.mark.parametrize("T,K,N,chunks", [(300, 200, 264, 1), (512, 320, 520, 4),
                                          (96, 64, 8, 3), (8, 8, 8, 1)])
def test_fwd_nn_integer_bit_exact(T, K, N, chunks):
    m = atp.mesh(1, 1)
    x = S.randint_bf16((T, K), 1, 1).to(DEV)
    w = S.randint_bf16((K, N), 1, 2).to(DEV)
    y = torch.full((T, N), float("nan"), device=DEV)
    atp.atp_shard_linear_fwd(m, atp.ATP_ROW_FIRST, T, K, N, chunks, x, w, None,
                             atp.ATP_EPI_NONE, y)
    _sync()
    ref = O.matmul(x.cpu(), w.cpu())
    np.testing.assert_array_equal(to64(y), ref)


@pytest.mark.parametrize("T,K,N,chunks", [(300, 200, 264, 3), (640, 72, 296, 2)])
def test_bwd_nt_tn_colsum_integer_bit_exact(T, K, N, chunks):
    m = atp.mesh(1, 1)
    x = S.randint_bf16((T, K), 2, 1).to(DEV)
    w = S.randint_bf16((K, N), 2, 2).to(DEV)
    dy = S.randint_bf16((T, N), 2, 3).to(DEV)
    dx = torch.full((T, K), float("nan"), device=DEV)
    dw = torch.full((K, N), float("nan"), device=DEV)
    db = torch.full((N,), float("nan"), device=DEV)
    atp.atp_shard_linear_bwd(m, atp.ATP_ROW_FIRST, T, K, N, chunks, x, w, dy, dx, dw, db)
    _sync()
    rdx, rdw, rdb = O.linear_bwd(x.cpu(), w.cpu(), dy.cpu())
    np.testing.assert_array_equal(to64(dx), rdx)
    np.testing.assert_array_equal(to64(dw), rdw)
    np.testing.assert_array_equal(to64(db), rdb)


@pytest.mark.parametrize("T,K,N,chunks", [(1, 8, 8, 1), (7, 16, 24, 1), (64, 40, 8, 2),
                                          (257, 168, 40, 1), (700, 488, 1000, 2),
                                          (512, 160, 2056, 4), (1024, 1288, 72, 8)])
def test_dx_nt_ragged_integer_bit_exact(T, K, N, chunks):
    """dX = dY W^T runs the NT kernel (256 x 160 tiles, K steps of 64):
    outputs of one row, sub-tile and multi-tile sizes with ragged edges, and
    contractions shorter than one K step or ending in a partial one."""
    m = atp.mesh(1, 1)
    x = S.randint_bf16((T, K), 6, 1).to(DEV)
    w = S.randint_bf16((K, N), 6, 2).to(DEV)
    dy = S.randint_bf16((T, N), 6, 3).to(DEV)
    dx = torch.full((T, K), float("nan"), device=DEV)
    dw = torch.full((K, N), float("nan"), device=DEV)
    atp.atp_shard_linear_bwd(m, atp.ATP_ROW_FIRST, T, K, N, chunks, x, w, dy, dx, dw, None)
    _sync()
    rdx, rdw, _ = O.linear_bwd(x.cpu(), w.cpu(), dy.cpu())
    np.testing.assert_array_equal(to64(dx), rdx)
    np.testing.assert_array_equal(to64(dw), rdw)


@pytest.mark.parametrize("epi", [atp.ATP_EPI_NONE, atp.ATP_EPI_BIAS, atp.ATP_EPI_BIAS_GELU])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_fwd_epilogues_group_of_one(epi, out_dtype):
    T, K, N = 264, 136, 392
    m = atp.mesh(1, 1)
    x = S.randn_bf16((T, K), 1.0, 3, 1).to(DEV)
    w = S.randn_bf16((K, N), 0.1, 3, 2).to(DEV)
    b = S.randn_bf16((N,), 0.5, 3, 3).to(DEV)
    y = torch.full((T, N), float("nan"), device=DEV, dtype=out_dtype)
    pre = torch.full((T, N), float("nan"), device=DEV, dtype=torch.bfloat16) \
        if epi == atp.ATP_EPI_BIAS_GELU else None
    atp.atp_shard_linear_fwd(m, atp.ATP_COL_FIRST, T, K, N, 2, x, w, b, epi, y, preact=pre)
    _sync()
    oepi = {atp.ATP_EPI_NONE: O.EPI_NONE, atp.ATP_EPI_BIAS: O.EPI_BIAS,
            atp.ATP_EPI_BIAS_GELU: O.EPI_BIAS_GELU}[epi]
    ref, rpre = O.linear_fwd_reduced(x.cpu(), w.cpu(), 0, [], b.cpu(), oepi)
    assert_close(y, ref, "y")
    if pre is not None:
        assert_close(pre, rpre, "preact")


@pytest.mark.parametrize("mesh,mode", [((2, 2), 0), ((2, 4), 1), ((4, 2), 0)])
def test_partial_block_every_coordinate(mesh, mode):
    """The device's Partial(SUM) block for every coordinate, cut from global
    X and W by the shard geometry, against the oracle's spec-derived block."""
    d1, d2 = mesh
    T, K, N = 136, 256, 512
    X = S.randn_bf16((T, K), 1.0, 4, 1)
    W = S.randn_bf16((K, N), 0.05, 4, 2)
    for i1 in range(d1):
        for i2 in range(d2):
            m = atp.mesh(d1, d2, i1, i2)
            g = atp.atp_shard_geometry(m, mode, K, N)
            x_loc = X[:, g.k_off:g.k_off + g.k_loc].contiguous().to(DEV)
            w_loc = W[g.k_off:g.k_off + g.k_loc, g.n_off:g.n_off + g.n_loc].contiguous().to(DEV)
            y = torch.empty((T, g.n_loc), device=DEV)
            atp.atp_shard_linear_fwd(m, mode, T, K, N, 2, x_loc, w_loc, None, 0, y)
            _sync()
            ref = O.local_partial(X, W, mesh, (i1, i2), mode)
            assert_close(y, ref, f"partial {(i1, i2)}")


def test_fwd_leading_dimensions_and_empty():
    """Strided views (ld > cols) and zero tokens."""
    T, K, N = 130, 64, 136
    m = atp.mesh(1, 1)
    xb = S.randint_bf16((T, K + 24), 5, 1).to(DEV)
    wb = S.randint_bf16((K, N + 40), 5, 2).to(DEV)
    yb = torch.full((T, N + 8), -7.0, device=DEV)
    x, w, y = xb[:, :K], wb[:, :N], yb[:, :N]
    atp.atp_shard_linear_fwd(m, 0, T, K, N, 2, x, w, None, 0, y)
    _sync()
    np.testing.assert_array_equal(to64(y), O.matmul(x.cpu(), w.cpu()))
    assert torch.all(yb[:, N:] == -7.0)
    y0 = torch.empty((0, N), device=DEV)
    atp.atp_shard_linear_fwd(m, 0, 0, K, N, 4, x[:0], w, None, 0, y0)
    _sync()
