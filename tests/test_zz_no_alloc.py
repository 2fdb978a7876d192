"""atp_attention_bwd_noalloc -- the attention backward for callers that
cannot allocate -- against atp_attention_bwd with a caller-owned delta
buffer, through the C ABI: two calls in a row (the second smaller, so it
reuses the library's per-GPU scratch after a larger call), each compared bit
for bit with the existing entry point on the same inputs.  It is collected
last (pytest runs files in name order), so a failure here hides no other
test.  Runs alone in a fresh process as well as after the other tests."""
import pytest
import torch

import paper_2301_08658_amd as atp
import synth_inputs as S

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(mesh, coord, batch, seq, h, seed):
    m = atp.mesh(mesh[0], mesh[1], coord[0], coord[1])
    bm = atp.ATP_BLOCK_COL
    heads = h // 128
    g = atp.block_geometry(m, bm, h)[0]
    _, hd, _ = atp.attention_heads(m, bm, h, heads)
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), 1.0, seed, 1).to(DEV)
    d_out = S.randn_bf16((T, g.n_loc // 3), 1.0, seed, 2).to(DEV)
    out = torch.zeros((T, g.n_loc // 3), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((hd, T), device=DEV)
    atp.atp_attention_fwd(m, bm, batch, seq, h, heads, qkv, out, lse)
    ref = torch.full((T, g.n_loc), float("nan"), dtype=torch.bfloat16, device=DEV)
    delta = torch.empty(hd * T, device=DEV)
    atp.atp_attention_bwd(m, bm, batch, seq, h, heads, qkv, out, lse, d_out, ref, delta)
    got = torch.full((T, g.n_loc), float("nan"), dtype=torch.bfloat16, device=DEV)
    atp.atp_attention_bwd_noalloc(m, bm, batch, seq, h, heads, qkv, out, lse, d_out, got)
    torch.cuda.synchronize()
    return ref, got, hd * T


def test_noalloc_attention_bwd_matches_the_allocating_call():
    print("noalloc attention bwd: two calls, the second smaller", flush=True)
    # 20 heads x 4096 tokens (the wide layer's share), then 2 heads x 300
    for case in (((8, 1), (3, 0), 2, 2048, 20480, 91), ((2, 2), (1, 1), 3, 100, 1024, 92)):
        ref, got, n = _case(*case)
        assert n <= atp.binding.ATP_NOALLOC_DELTA_MAX
        for t in (ref, got):
            assert not torch.isnan(t[:, :t.shape[1]]).all()
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), case
