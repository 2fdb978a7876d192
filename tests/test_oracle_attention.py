"""Pins of the oracle's attention core (Sec. 2.1 Formula (mha) with a causal
mask; Sec. 3.2.1's scatter of the attention heads), independent of the
oracle's own code:

* torch float64 scaled_dot_product_attention and its autograd (a library
  routine) on random inputs, lse against torch's logsumexp of the masked
  scores;
* closed forms: q = 0 gives uniform weights, so o[t] is the mean of v[0..t]
  and lse[t] = log(t + 1); one token gives o = v;
* invariants: causality (later keys and values never change earlier rows),
  sum over keys of dK is zero (softmax rows sum to one), central finite
  differences of a scalar loss;
* the scatter: the members of a group attend over disjoint runs of heads
  that together cover the block, and concatenated they equal the attention
  of the whole block."""
import numpy as np
import pytest
import torch

import oracle as O


def _rand(rng, *shape):
    return rng.standard_normal(shape)


@pytest.mark.parametrize("S,d", [(1, 8), (5, 4), (37, 16), (64, 32), (130, 8)])
def test_attention_matches_torch_float64(S, d):
    rng = np.random.default_rng(S * 100 + d)
    q, k, v, do = (_rand(rng, S, d) for _ in range(4))
    o, lse = O.attention_fwd(q, k, v)
    qt, kt, vt = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    ot = torch.nn.functional.scaled_dot_product_attention(qt[None], kt[None], vt[None],
                                                          is_causal=True)[0]
    np.testing.assert_allclose(o, ot.detach().numpy(), rtol=0, atol=1e-12)
    scores = (qt @ kt.T).detach() / np.sqrt(d)
    scores = scores.masked_fill(torch.triu(torch.ones(S, S, dtype=torch.bool), 1), -np.inf)
    np.testing.assert_allclose(lse, torch.logsumexp(scores, dim=1).numpy(), rtol=0, atol=1e-12)
    ot.backward(torch.tensor(do))
    dq, dk, dv = O.attention_bwd(q, k, v, do)
    for got, ref in ((dq, qt.grad), (dk, kt.grad), (dv, vt.grad)):
        np.testing.assert_allclose(got, ref.numpy(), rtol=0, atol=1e-11)


def test_attention_zero_queries_give_prefix_means():
    rng = np.random.default_rng(3)
    S, d = 50, 8
    k, v = _rand(rng, S, d), _rand(rng, S, d)
    o, lse = O.attention_fwd(np.zeros((S, d)), k, v)
    prefix = np.cumsum(v, axis=0) / np.arange(1, S + 1)[:, None]
    np.testing.assert_allclose(o, prefix, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, np.log(np.arange(1, S + 1)), rtol=0, atol=1e-13)


def test_attention_one_token():
    rng = np.random.default_rng(4)
    q, k, v = (_rand(rng, 1, 6) for _ in range(3))
    o, lse = O.attention_fwd(q, k, v)
    np.testing.assert_allclose(o, v, rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse, [(q @ k.T)[0, 0] / np.sqrt(6)], rtol=0, atol=1e-15)


def test_attention_is_causal():
    rng = np.random.default_rng(5)
    S, d = 40, 8
    q, k, v = (_rand(rng, S, d) for _ in range(3))
    o, _ = O.attention_fwd(q, k, v)
    k2, v2 = k.copy(), v.copy()
    k2[25:] += 3.0
    v2[25:] -= 2.0
    o2, _ = O.attention_fwd(q, k2, v2)
    np.testing.assert_array_equal(o[:25], o2[:25])
    assert np.abs(o[25:] - o2[25:]).max() > 1e-3


def test_attention_key_gradients_sum_to_zero():
    # each softmax row sums to one, so its scores' gradients sum to zero over
    # the keys, and so does dK = dS^T q / sqrt(d) summed over the keys
    rng = np.random.default_rng(6)
    S, d = 33, 8
    q, k, v, do = (_rand(rng, S, d) for _ in range(4))
    _, dk, _ = O.attention_bwd(q, k, v, do)
    np.testing.assert_allclose(dk.sum(axis=0), 0.0, rtol=0, atol=1e-12)


def test_attention_gradients_match_finite_differences():
    rng = np.random.default_rng(7)
    S, d = 6, 3
    q, k, v, w = (_rand(rng, S, d) for _ in range(4))

    def loss(q_, k_, v_):
        return float((O.attention_fwd(q_, k_, v_)[0] * w).sum())

    dq, dk, dv = O.attention_bwd(q, k, v, w)
    eps = 1e-6
    for which, grad in ((0, dq), (1, dk), (2, dv)):
        for (i, j) in [(0, 0), (2, 1), (5, 2), (3, 0)]:
            args = [q.copy(), k.copy(), v.copy()]
            args[which][i, j] += eps
            up = loss(*args)
            args[which][i, j] -= 2 * eps
            dn = loss(*args)
            assert abs((up - dn) / (2 * eps) - grad[i, j]) < 1e-7, (which, i, j)


@pytest.mark.parametrize("group", [1, 2, 4])
def test_scatter_over_group_covers_the_block(group):
    """Members 0..g-1 of the reduction group take disjoint head runs; their
    outputs side by side are the attention of every head of the block."""
    rng = np.random.default_rng(8 + group)
    batch, seq, hd, heads = 2, 9, 4, 4
    qkv = _rand(rng, batch * seq, 3 * hd * heads)
    whole, lse_whole = O.attention_core_local(qkv, batch, seq, hd, 1, 0)
    parts, lses, firsts = [], [], []
    for j in range(group):
        h0, n = O.attention_heads(qkv.shape[1], hd, group, j)
        firsts.append((h0, n))
        o, lse = O.attention_core_local(qkv, batch, seq, hd, group, j)
        parts.append(o)
        lses.append(lse)
    assert [f[0] for f in firsts] == [j * heads // group for j in range(group)]
    np.testing.assert_array_equal(np.concatenate(parts, axis=1), whole)
    np.testing.assert_array_equal(np.concatenate(lses, axis=0), lse_whole)
    # head j of the block is attention over its own [q | k | v] columns
    j = heads - 1
    c = 3 * hd * j
    o, _ = O.attention_fwd(qkv[:seq, c:c + hd], qkv[:seq, c + hd:c + 2 * hd],
                           qkv[:seq, c + 2 * hd:c + 3 * hd])
    np.testing.assert_array_equal(whole[:seq, j * hd:(j + 1) * hd], o)


def test_scatter_backward_matches_per_head_backward():
    rng = np.random.default_rng(9)
    batch, seq, hd, heads = 2, 7, 4, 4
    qkv = _rand(rng, batch * seq, 3 * hd * heads)
    do = _rand(rng, batch * seq, 2 * hd)
    dqkv = O.attention_core_bwd_local(qkv, do, batch, seq, hd, 2, 1)   # heads 2, 3
    for jj, head in enumerate((2, 3)):
        c = 3 * hd * head
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            dq, dk, dv = O.attention_bwd(qkv[r, c:c + hd], qkv[r, c + hd:c + 2 * hd],
                                         qkv[r, c + 2 * hd:c + 3 * hd],
                                         do[r, jj * hd:(jj + 1) * hd])
            got = dqkv[r, 3 * hd * jj:3 * hd * (jj + 1)]
            np.testing.assert_array_equal(got, np.concatenate([dq, dk, dv], axis=1))


def test_attention_block_matches_torch_autograd():
    """The unsharded attention block (QKV -> causal core -> out-proj) and
    every gradient against torch float64: the core as
    scaled_dot_product_attention(is_causal=True) per head and autograd through
    the whole chain (library routines).  Pins the [q | k | v] column order of
    each head, the heads' side-by-side order in A, the biases and the
    gradients the chained backward produces."""
    rng = np.random.default_rng(21)
    batch, seq, d, heads = 2, 6, 4, 3
    h, T = d * heads, 2 * 6
    X = rng.standard_normal((T, h))
    Wq, bq = rng.standard_normal((h, 3 * h)) * 0.4, rng.standard_normal(3 * h) * 0.1
    Wo, bo = rng.standard_normal((h, h)) * 0.4, rng.standard_normal(h) * 0.1
    dO = rng.standard_normal((T, h))
    f = O.attention_block_global(X, Wq, bq, Wo, bo, batch, seq, d)
    g = O.attention_block_global_bwd(X, Wq, Wo, f, dO, batch, seq, d)

    t = {k: torch.tensor(v, requires_grad=True) for k, v in
         dict(X=X, Wq=Wq, bq=bq, Wo=Wo, bo=bo).items()}
    qkv = t["X"] @ t["Wq"] + t["bq"]
    qkv.retain_grad()
    q, k, v = qkv.view(batch, seq, heads, 3, d).permute(3, 0, 2, 1, 4).unbind(0)
    a = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
    A = a.permute(0, 2, 1, 3).reshape(T, h)
    A.retain_grad()
    o = A @ t["Wo"] + t["bo"]
    (o * torch.tensor(dO)).sum().backward()
    scores = (q @ k.transpose(-1, -2)) / np.sqrt(d)
    scores = scores.masked_fill(torch.triu(torch.ones(seq, seq, dtype=torch.bool), 1), -np.inf)
    lse = torch.logsumexp(scores, -1).permute(1, 0, 2).reshape(heads, T)

    close = lambda a_, b_: np.testing.assert_allclose(a_, b_.detach().numpy(), rtol=1e-10,  # noqa
                                                      atol=1e-12)
    close(f["qkv"], qkv)
    close(f["attn"], A)
    close(f["o"], o)
    close(f["lse"], lse)
    close(g["d_attn"], A.grad)
    close(g["d_qkv"], qkv.grad)
    close(g["dx"], t["X"].grad)
    close(g["dw_qkv"], t["Wq"].grad)
    close(g["db_qkv"], t["bq"].grad)
    close(g["dw_out"], t["Wo"].grad)
    close(g["db_out"], t["bo"].grad)
