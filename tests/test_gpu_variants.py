"""Variants of one reduced shard linear (Sec. 3.2) beside the chunked overlap
of Sec. 4.1:

* the reduction fused into the GEMM's epilogue (one launch, the own partial
  never stored): the design Sec. 4.1 contrasts chunking with.  Its terms are
  summed in group order, so it must equal the GEMM + chunked reduction bit
  for bit, and the oracle within tolerance;
* bf16 Partial(SUM) blocks (Sec. 5 trains in 16-bit and all-reduces 16-bit
  activations): each member's partial rounded to bf16, the group's values
  summed in fp32.  The oracle is its reduction of the bf16-rounded partials;
  with small integer inputs every step is exact and the bits must match."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_08658_amd as atp
import synth_inputs as S
from helpers import DEV, assert_close, to64

pytestmark = pytest.mark.gpu

OEPI = {atp.ATP_EPI_NONE: O.EPI_NONE, atp.ATP_EPI_BIAS: O.EPI_BIAS,
        atp.ATP_EPI_BIAS_GELU: O.EPI_BIAS_GELU}

# (mode, mesh, coord, tokens, k, n, chunks, epi, out dtype)
CASES = [(atp.ATP_ROW_FIRST, (4, 2), (2, 1), 256, 1024, 512, 2, atp.ATP_EPI_BIAS,
          torch.bfloat16),
         (atp.ATP_COL_FIRST, (2, 4), (1, 3), 384, 1024, 2048, 3, atp.ATP_EPI_BIAS_GELU,
          torch.bfloat16),
         (atp.ATP_ROW_FIRST, (8, 1), (5, 0), 200, 2048, 640, 2, atp.ATP_EPI_NONE, torch.float32),
         (atp.ATP_ROW_FIRST, (8, 1), (0, 0), 520, 4096, 1280, 4, atp.ATP_EPI_BIAS,
          torch.float32)]
IDS = [f"m{c[0]}_{c[1][0]}x{c[1][1]}_e{c[7]}_{'bf16' if c[8] == torch.bfloat16 else 'f32'}"
       for c in CASES]


def _inputs(case, seed, integer=False):
    mode, mesh, coord, T, k, n, chunks, epi, odt = case
    m = atp.mesh(mesh[0], mesh[1], coord[0], coord[1])
    g = atp.atp_shard_geometry(m, mode, k, n)
    if integer:
        x = S.randint_bf16((T, g.k_loc), seed, 1, -1, 1).to(DEV)
        w = S.randint_bf16((g.k_loc, g.n_loc), seed, 2, -1, 1).to(DEV)
        peers = [S.randint_f32((T, g.n_loc), seed, 10 + j, -64, 64).to(DEV)
                 for j in range(g.red_size)]
        bias = S.randint_bf16((g.n_loc,), seed, 3, -2, 2).to(DEV)
    else:
        x = S.randn_bf16((T, g.k_loc), 1.0, seed, 1).to(DEV)
        w = S.randn_bf16((g.k_loc, g.n_loc), 0.02, seed, 2).to(DEV)
        sp = S.peer_sigma(g.k_loc, 0.02, 1.0)
        peers = [S.randn_f32((T, g.n_loc), sp, seed, 10 + j).to(DEV) for j in range(g.red_size)]
        bias = S.randn_bf16((g.n_loc,), 0.02, seed, 3).to(DEV)
    return m, g, x, w, peers, bias


def _pipeline(case, m, g, x, w, peers, bias):
    """GEMM chunks into the own slot, then the chunked reduction (one stream)."""
    mode, mesh, coord, T, k, n, chunks, epi, odt = case
    tab = list(peers)
    tab[g.red_index] = torch.empty((T, g.n_loc), dtype=torch.float32, device=DEV)
    atp.atp_shard_linear_fwd(m, mode, T, k, n, chunks, x, w, None, atp.ATP_EPI_NONE,
                             tab[g.red_index])
    out = torch.full((T, g.n_loc), 3.0, dtype=odt, device=DEV)
    pre = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=DEV) \
        if epi == atp.ATP_EPI_BIAS_GELU else None
    atp.atp_chunked_partial_reduce(g.red_size, T, g.n_loc, chunks, tab,
                                   bias if epi != atp.ATP_EPI_NONE else None, epi, out,
                                   preact_out=pre)
    return out, pre, tab[g.red_index]


def _fused(case, m, g, x, w, peers, bias):
    mode, mesh, coord, T, k, n, chunks, epi, odt = case
    out = torch.full((T, g.n_loc), 5.0, dtype=odt, device=DEV)
    pre = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=DEV) \
        if epi == atp.ATP_EPI_BIAS_GELU else None
    pp = [None if j == g.red_index else p for j, p in enumerate(peers)]
    atp.atp_shard_linear_fwd_fused(m, mode, T, k, n, x, w, pp,
                                   bias if epi != atp.ATP_EPI_NONE else None, epi, out, pre)
    return out, pre


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_fused_equals_gemm_then_reduction(case):
    print(f"fused vs pipeline {case}", flush=True)
    m, g, x, w, peers, bias = _inputs(case, 81)
    ref, ref_pre, _ = _pipeline(case, m, g, x, w, peers, bias)
    out, pre = _fused(case, m, g, x, w, peers, bias)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    if pre is not None:
        assert torch.equal(pre, ref_pre)


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_fused_matches_oracle(case):
    print(f"fused oracle {case}", flush=True)
    m, g, x, w, peers, bias = _inputs(case, 82)
    epi = case[7]
    out, pre = _fused(case, m, g, x, w, peers, bias)
    torch.cuda.synchronize()
    others = [p.cpu() for j, p in enumerate(peers) if j != g.red_index]
    ref, rpre = O.linear_fwd_reduced(x.cpu(), w.cpu(), g.red_index, others,
                                     bias.cpu() if epi != atp.ATP_EPI_NONE else None, OEPI[epi])
    assert_close(out, ref, "fused out")
    if pre is not None:
        assert_close(pre, rpre, "fused preact")


def test_fused_integer_exact_and_group_of_one():
    case = CASES[3]
    m, g, x, w, peers, bias = _inputs(case, 83, integer=True)
    out, _ = _fused(case, m, g, x, w, peers, bias)
    torch.cuda.synchronize()
    others = [p.cpu() for j, p in enumerate(peers) if j != g.red_index]
    ref, _ = O.linear_fwd_reduced(x.cpu(), w.cpu(), g.red_index, others, bias.cpu(), O.EPI_BIAS)
    np.testing.assert_array_equal(to64(out), ref)
    # a group of one: the plain GEMM with its epilogue
    m1 = atp.mesh(1, 1, 0, 0)
    T, k, n = 256, 512, 384
    x1 = S.randn_bf16((T, k), 1.0, 84, 1).to(DEV)
    w1 = S.randn_bf16((k, n), 0.02, 84, 2).to(DEV)
    b1 = S.randn_bf16((n,), 0.02, 84, 3).to(DEV)
    a = torch.empty((T, n), dtype=torch.bfloat16, device=DEV)
    b = torch.empty_like(a)
    pa = torch.empty_like(a)
    pb = torch.empty_like(a)
    atp.atp_shard_linear_fwd_fused(m1, atp.ATP_ROW_FIRST, T, k, n, x1, w1, [None], b1,
                                   atp.ATP_EPI_BIAS_GELU, a, pa)
    atp.atp_shard_linear_fwd(m1, atp.ATP_ROW_FIRST, T, k, n, 1, x1, w1, b1,
                             atp.ATP_EPI_BIAS_GELU, b, pb)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(pa, pb)


def test_fused_errors():
    case = CASES[0]
    m, g, x, w, peers, bias = _inputs(case, 85)
    mode, mesh, coord, T, k, n, chunks, epi, odt = case
    out = torch.empty((T, g.n_loc), dtype=odt, device=DEV)
    pp = [None if j == g.red_index else p for j, p in enumerate(peers)]
    pp[(g.red_index + 1) % g.red_size] = None            # a missing peer
    with pytest.raises(atp.AtpError):
        atp.atp_shard_linear_fwd_fused(m, mode, T, k, n, x, w, pp, bias, epi, out)
    m16 = atp.mesh(16, 1, 0, 0)                          # group of 16 > 8
    g16 = atp.atp_shard_geometry(m16, atp.ATP_ROW_FIRST, 2048, 256)
    x16 = torch.zeros((64, g16.k_loc), dtype=torch.bfloat16, device=DEV)
    w16 = torch.zeros((g16.k_loc, 256), dtype=torch.bfloat16, device=DEV)
    p16 = [None] + [torch.zeros((64, 256), device=DEV) for _ in range(15)]
    with pytest.raises(atp.AtpError):
        atp.atp_shard_linear_fwd_fused(m16, atp.ATP_ROW_FIRST, 64, 2048, 256, x16, w16, p16,
                                       None, atp.ATP_EPI_NONE,
                                       torch.empty((64, 256), device=DEV))


def _bf16_pipeline(case, m, g, x, w, peers16, bias):
    mode, mesh, coord, T, k, n, chunks, epi, odt = case
    tab = list(peers16)
    tab[g.red_index] = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=DEV)
    atp.atp_shard_linear_fwd(m, mode, T, k, n, chunks, x, w, None, atp.ATP_EPI_NONE,
                             tab[g.red_index])
    out = torch.full((T, g.n_loc), 3.0, dtype=odt, device=DEV)
    pre = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=DEV) \
        if epi == atp.ATP_EPI_BIAS_GELU else None
    atp.atp_chunked_partial_reduce_bf16(g.red_size, T, g.n_loc, chunks, tab,
                                        bias if epi != atp.ATP_EPI_NONE else None, epi, out,
                                        preact_out=pre)
    return out, pre, tab[g.red_index]


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_bf16_partials_match_oracle(case):
    print(f"bf16 partials {case}", flush=True)
    m, g, x, w, peers, bias = _inputs(case, 86)
    epi = case[7]
    peers16 = [p.to(torch.bfloat16) for p in peers]
    out, pre, own = _bf16_pipeline(case, m, g, x, w, peers16, bias)
    torch.cuda.synchronize()
    own_ref = O.matmul(x.cpu(), w.cpu())
    # the own partial is the product rounded once to bf16
    assert_close(own, O.round_bf16(own_ref), "own bf16 partial")
    parts = [p.cpu() for p in peers16]
    parts[g.red_index] = O.round_bf16(own_ref)
    ref, rpre = O.partial_reduce(parts, bias.cpu() if epi != atp.ATP_EPI_NONE else None,
                                 OEPI[epi])
    assert_close(out, ref, "out")
    if pre is not None:
        assert_close(pre, rpre, "preact")


def test_bf16_partials_integer_exact():
    """x, w in {-1, 0, 1} over k_loc = 256: every partial is an integer of
    magnitude <= 256, exact in bf16, and the group's sum is exact in fp32,
    so the own bf16 partial and the reduced output match the oracle's exact
    values bit for bit."""
    case = (atp.ATP_ROW_FIRST, (8, 1), (3, 0), 256, 2048, 512, 2, atp.ATP_EPI_BIAS, torch.float32)
    m, g, x, w, _, bias = _inputs(case, 87, integer=True)
    assert g.k_loc == 256
    peers16 = [S.randint_bf16((case[3], g.n_loc), 87, 20 + j, -100, 100).to(DEV)
               for j in range(g.red_size)]
    out, _, own = _bf16_pipeline(case, m, g, x, w, peers16, bias)
    torch.cuda.synchronize()
    own_ref = O.matmul(x.cpu(), w.cpu())
    np.testing.assert_array_equal(to64(own), own_ref)
    parts = [p.cpu() for p in peers16]
    parts[g.red_index] = own_ref
    ref, _ = O.partial_reduce(parts, bias.cpu(), O.EPI_BIAS)
    np.testing.assert_array_equal(to64(out), ref)
