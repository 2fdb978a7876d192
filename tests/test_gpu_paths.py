"""The bf16 transpose kernel, and the block calls with a workspace against
the same calls without one.

With a workspace the forward runs from W^T and dW from X^T and dY^T (both
operands contiguous along k); without one they read W, X and dY as given
(transposing LDS reads).  Both layouts sum each element's products in the
same order, so the paths give the same bits, except that with a workspace
chunk products with too few output tiles to fill the chip are split over k,
which sums in a different order: there the paths agree to fp32 rounding,
and a bf16 output differs by at most a couple of units in the last place
where the two fp32 values straddle a rounding boundary.  fc1's dW and db are
token sums of the bf16 dh_pre, which may sit one unit apart between the
paths, so they get a looser bound.  Where no product splits (the wide 8 x 1
layer) the paths agree bit for bit.  Both paths are checked against the
oracle elsewhere."""
import pytest
import torch

import paper_2301_08658_amd as atp
import synth_inputs as S
from helpers import assert_paths_agree, make_block_inputs, run_block_bwd, run_block_fwd

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def bits(t):
    return t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32)


@pytest.mark.parametrize("rows,cols,pad_s,pad_d", [
    (1, 8, 0, 0), (7, 16, 8, 0), (64, 64, 0, 8), (65, 72, 0, 0), (300, 200, 16, 24),
    (513, 1032, 8, 8), (4096, 2560, 0, 0), (2, 4104, 0, 8),
    # multiples of 8 (the register-block kernel), with partial 64 x 256 tiles
    (8, 8, 0, 0), (72, 264, 8, 8), (4104, 520, 0, 8), (136, 2056, 16, 0)])
def test_transpose_matches_torch(rows, cols, pad_s, pad_d):
    print(f"transpose {rows}x{cols} pads {pad_s},{pad_d}", flush=True)
    src_full = S.randint_bf16((rows, cols + pad_s), 7, 901).to(DEV)
    src = src_full[:, :cols]
    ldd = ((rows + 7) // 8) * 8 + pad_d
    dst_full = torch.full((cols, ldd), -1.0, dtype=torch.bfloat16, device=DEV)
    atp.atp_transpose_bf16(src, dst_full[:, :rows])
    torch.cuda.synchronize()
    assert torch.equal(bits(dst_full[:, :rows]), bits(src.t().contiguous()))
    if ldd > rows:   # the padding columns are left alone
        assert torch.all(dst_full[:, rows:] == -1.0)


def test_transpose_empty_and_errors():
    z = torch.empty((0, 8), dtype=torch.bfloat16, device=DEV)
    atp.atp_transpose_bf16(z, torch.empty((8, 0), dtype=torch.bfloat16, device=DEV))
    a = torch.zeros((16, 16), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(atp.AtpError):
        atp.atp_transpose_bf16(a, a)            # in place is not supported


CASES = [  # (mode, mesh, coord, T, h, chunks)
    ("col", (2, 2), (1, 0), 256, 512, 2),
    ("col", (2, 4), (1, 3), 512, 1024, 4),
    ("row", (4, 2), (3, 1), 512, 1024, 4),
    ("col", (1, 1), (0, 0), 128, 256, 1),
    ("col", (8, 1), (7, 0), 256, 2048, 2),
    ("col", (2, 2), (0, 1), 200, 512, 2),     # tokens % 8 == 0, not a tile multiple
    ("row", (2, 2), (1, 1), 132, 512, 2),     # tokens % 8 != 0: dW falls back to TN
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}{c[1][0]}x{c[1][1]}_T{c[3]}")
def test_block_forward_workspace_equals_direct(case):
    mode, mesh, coord, T, h, chunks = case
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=21, on_device=True)
    print(f"fwd {case}", flush=True)
    a = run_block_fwd(inp, chunks)
    b = run_block_fwd(inp, chunks, workspace=True)
    torch.cuda.synchronize()
    for k in ("qkv", "o", "h", "pre", "z"):
        assert_paths_agree(a[k], b[k], k)
    for i, (x, y) in enumerate(zip(a["own"], b["own"])):
        if x is not None:
            assert_paths_agree(x, y, f"partial {i}")


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}{c[1][0]}x{c[1][1]}_T{c[3]}")
def test_block_backward_workspace_equals_direct(case):
    mode, mesh, coord, T, h, chunks = case
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=22, on_device=True, bwd=True)
    print(f"bwd {case}", flush=True)
    a = run_block_bwd(inp, chunks)
    b = run_block_bwd(inp, chunks, workspace=True)
    torch.cuda.synchronize()
    _check_bwd_paths(a, b)


def _check_bwd_paths(a, b):
    for k in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
        assert_paths_agree(a[k], b[k], k)
    for i in range(4):
        rel = 2e-3 if i == 2 else 1e-4
        assert_paths_agree(a["dw"][i], b["dw"][i], f"dw {i}", rel)
        assert_paths_agree(a["db"][i], b["db"][i], f"db {i}", rel)


def test_benchmark_workload_workspace_equals_direct():
    """No chunk product of the wide 8 x 1 layer splits: bit for bit."""
    w = S.WORKLOADS["wide_h20480_col_8x1"]
    inp = make_block_inputs(w["mode"], w["mesh"], (0, 0), w["tokens"], w["h"], w["sigma_w"],
                            seed=23, on_device=True, bwd=True)
    print("bench workload fwd+bwd, both paths", flush=True)
    fa = run_block_fwd(inp, w["chunks"])
    fb = run_block_fwd(inp, w["chunks"], workspace=True)
    ba = run_block_bwd(inp, w["chunks"])
    bb = run_block_bwd(inp, w["chunks"], workspace=True)
    torch.cuda.synchronize()
    for k in ("qkv", "o", "h", "pre", "z"):
        assert torch.equal(bits(fa[k]), bits(fb[k])), k
    for k in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
        assert torch.equal(bits(ba[k]), bits(bb[k])), k
    for i in range(4):
        assert torch.equal(bits(ba["dw"][i]), bits(bb["dw"][i])), f"dw {i}"
        assert torch.equal(bits(ba["db"][i]), bits(bb["db"][i])), f"db {i}"
