"""Split-K of the chunked products that feed a reduction (workspace path).

A chunk's product with too few 256 x 160 tiles to fill the chip is split over
its contraction: each split writes an fp32 slab, and the slabs are summed in
split order into the device's own partial buffer before the chunk's
reduction reads it.  The split plan is a function of the chunk's shape.

* the split kernels run where the plan asks for them (the library's profile),
* results match the oracle, with odd split counts and a shorter last split,
* with integer-valued inputs every partial sum is exact, so the own partials
  and the reduced outputs match the oracle bit for bit,
* repeated calls give the same bits.
Full-size configurations with splits are checked in the workload tests."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_08658_amd as atp
from helpers import (LIN, assert_close, check_bwd, check_fwd, make_block_inputs,
                     oracle_block_bwd, oracle_block_fwd, run_block_bwd, run_block_fwd, to64)

pytestmark = pytest.mark.gpu

# (mode, mesh, coord, tokens, h, chunks): h = 2000 gives contractions of 1000,
# 3000 and 4000 (split 4, 12 and 16 ways with a shorter last split); h = 2048
# on 2 x 4 splits fc2's 4096 13 ways of 320
CASES = [("col", (2, 2), (1, 0), 256, 2000, 2),
         ("row", (2, 2), (0, 1), 256, 2000, 2),
         ("col", (2, 4), (1, 2), 1024, 2048, 2)]
IDS = [f"{c[0]}{c[1][0]}x{c[1][1]}_h{c[4]}" for c in CASES]


def _profiled_names(fn):
    atp.atp_profile_enable(2)
    try:
        fn()
        torch.cuda.synchronize()
        recs = atp.atp_profile_collect(256)
    finally:
        atp.atp_profile_enable(0)
    return [r["name"] if isinstance(r, dict) else r[0] for r in recs]


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_split_kernels_run_on_workspace_path_only(case):
    mode, mesh, coord, T, h, chunks = case
    print(f"splitk plan {case}", flush=True)
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=41, bwd=True)
    for ws in (True, False):
        names = _profiled_names(lambda: (run_block_fwd(inp, chunks, workspace=ws),
                                         run_block_bwd(inp, chunks, workspace=ws)))
        split = [n for n in names if n.startswith("gemm_nt_splitk")]
        sums = [n for n in names if n.startswith("split_sum")]
        if ws:
            assert split and sums, names
        else:
            assert not split and not sums, names


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_split_forward_matches_oracle(case):
    mode, mesh, coord, T, h, chunks = case
    print(f"splitk fwd {case}", flush=True)
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=42)
    out = run_block_fwd(inp, chunks, workspace=True)
    torch.cuda.synchronize()
    check_fwd(out, *oracle_block_fwd(O, inp), what="split")
    for i, g in enumerate(inp["G"][:3]):
        if g.red_size > 1:
            xin = inp["a"] if i == 1 else inp["x"]
            assert_close(out["own"][i], O.matmul(xin.cpu(), inp["wkn"][i].cpu()),
                         f"own partial {LIN[i]}")


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_split_backward_matches_oracle(case):
    mode, mesh, coord, T, h, chunks = case
    print(f"splitk bwd {case}", flush=True)
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=43, bwd=True)
    out = run_block_bwd(inp, chunks, workspace=True)
    torch.cuda.synchronize()
    check_bwd(out, *oracle_block_bwd(O, inp), what="split")


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_split_integer_partials_bit_exact(case):
    """Integer inputs: each split's sum, the sum of the splits and the
    reduction are exact, so the own partials equal X W exactly and the
    reduced QKV / out-proj outputs are the oracle's values rounded once."""
    mode, mesh, coord, T, h, chunks = case
    print(f"splitk integer {case}", flush=True)
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.0, seed=44, integer=True)
    out = run_block_fwd(inp, chunks, workspace=True)
    torch.cuda.synchronize()
    ref, _ = oracle_block_fwd(O, inp)
    for i, g in enumerate(inp["G"][:3]):
        if g.red_size > 1:
            xin = inp["a"] if i == 1 else inp["x"]
            np.testing.assert_array_equal(to64(out["own"][i]),
                                          O.matmul(xin.cpu(), inp["wkn"][i].cpu()),
                                          err_msg=f"own partial {LIN[i]}")
    for key in ("qkv", "o"):
        np.testing.assert_array_equal(to64(out[key]), O.round_bf16(ref[key]), err_msg=key)


def test_split_repeated_calls_identical():
    mode, mesh, coord, T, h, chunks = CASES[0]
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=45, bwd=True)
    a = run_block_fwd(inp, chunks, workspace=True)
    b = run_block_fwd(inp, chunks, workspace=True)
    ba = run_block_bwd(inp, chunks, workspace=True)
    bb = run_block_bwd(inp, chunks, workspace=True)
    torch.cuda.synchronize()
    for key in ("qkv", "o", "h", "pre", "z"):
        assert torch.equal(a[key], b[key]), key
    for key in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
        assert torch.equal(ba[key], bb[key]), key
