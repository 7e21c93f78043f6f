"""Pins of the batch-padding reading of the oracle (Appendix "Padding and
Masking": batched sequences padded to a common length, m and b fixed for the
batch, so a short sequence can have whole key blocks of padding).

The reading: a block with no real key gets R = 0 and no L weight (Z_L =
-inf), rows beyond a sequence's length are zero in O.  What fixes it, beyond
the code that states it:
* b = 1 reduces MonarchAttention to exact softmax attention for every T
  (each block is one key); with padding that must be attention over the
  real keys only, which fails if an empty block kept any L weight;
* at T = 1 a query row's output depends on no other query row (alpha_R, c_R
  come from L^(0) = I), so a sequence with whole padded blocks must give the
  same real rows as the single-sequence problem with m = ceil(n / b);
* M stays row-stochastic, with zero columns at the padded keys;
* the two independent formulations (materialised factors in numpy, the
  state form in C) agree.
"""
import numpy as np
import pytest

import oracle
import oracle.naive as nv
import synth_inputs as si


def _qkv(B, H, N, d, seed, scale=1.5):
    q, k, v = si.random_qkv(B, H, N, d, "f32", seed=seed, scale=scale)
    return (x.astype(np.float64) for x in (q, k, v))


@pytest.mark.parametrize("T", [1, 2, 3])
def test_single_key_blocks_give_exact_attention_over_real_keys(oracle_lib, T):
    N, d = 12, 8
    q, k, v = _qkv(3, 2, N, d, seed=11)
    lens = np.array([5, 12, 1])
    for o in (oracle.monarch_attention_varlen(q, k, v, lens, N, 1, T),
              nv.monarch_attention_varlen(q, k, v, lens, N, 1, T)):
        for bi, n in enumerate(lens):
            for h in range(2):
                ref = nv.dense_softmax_attention(q[bi, h, :n], k[bi, h, :n], v[bi, h, :n])
                np.testing.assert_allclose(o[bi, h, :n], ref, rtol=0, atol=1e-13)
                assert np.all(o[bi, h, n:] == 0.0)


@pytest.mark.parametrize("n,m,b", [(5, 4, 3), (7, 4, 3), (9, 5, 4), (3, 6, 4), (16, 6, 4)])
def test_one_step_matches_the_problem_without_empty_blocks(oracle_lib, n, m, b):
    N = m * b
    q, k, v = _qkv(1, 2, N, 6, seed=20 + n)
    o = oracle.monarch_attention_varlen(q, k, v, np.array([n]), m, b, 1)
    m2 = -(-n // b)
    ref = oracle.monarch_attention(q[:, :, :n], k[:, :, :n], v[:, :, :n], m2, b, 1)
    np.testing.assert_allclose(o[:, :, :n], ref, rtol=0, atol=1e-13)
    assert np.all(o[:, :, n:] == 0.0)


def test_more_steps_depend_on_the_padded_query_rows(oracle_lib):
    """For T >= 2 the zero query rows of the empty blocks take part through c_R
    (the paper's padded rows are live), so the result differs from the problem
    with fewer blocks: the T = 1 equality above is not a general identity."""
    n, m, b = 5, 4, 3
    q, k, v = _qkv(1, 1, m * b, 6, seed=31)
    o = oracle.monarch_attention_varlen(q, k, v, np.array([n]), m, b, 2)
    ref = oracle.monarch_attention(q[:, :, :n], k[:, :, :n], v[:, :, :n], 2, b, 2)
    assert np.abs(o[:, :, :n] - ref).max() > 1e-6


@pytest.mark.parametrize("n,m,b,T", [(5, 4, 3, 2), (2, 4, 3, 3), (10, 4, 3, 2), (0, 3, 3, 2)])
def test_padded_monarch_is_row_stochastic_with_zero_padded_columns(n, m, b, T):
    q, k, _ = _qkv(1, 1, m * b, 5, seed=40 + n)
    L, R = nv.factors(q[0, 0, :n], k[0, 0, :n], m, b, T, n=n, batch_padding=True)
    M = nv.dense_monarch(L, R)
    assert np.all(M >= 0.0)
    assert np.all(M[:, n:] == 0.0)
    rows = M.sum(axis=1)
    np.testing.assert_allclose(rows, 1.0 if n > 0 else 0.0, rtol=0, atol=1e-13)


@pytest.mark.parametrize("m,b", [(4, 3), (3, 5)])
def test_padded_ascent(m, b):
    """f(M) never decreases over the half-steps: each update stays the exact block
    maximiser over the matrices whose padded columns are zero."""
    n = b + 1  # one partial block, the rest padding
    q, k, _ = _qkv(1, 1, m * b, 5, seed=50 + m)
    L, R, hist = nv.factors(q[0, 0, :n], k[0, 0, :n], m, b, 3, n=n, batch_padding=True, history=True)
    qp, kp = nv.pad_rows(q[0, 0, :n], m, b), nv.pad_rows(k[0, 0, :n], m, b)
    vals = [nv.objective_dense(nv.dense_monarch(Lh, Rh), qp, kp) for Lh, Rh in hist[1:]]
    assert all(b2 >= a2 - 1e-12 for a2, b2 in zip(vals, vals[1:]))


@pytest.mark.parametrize("m,b,T", [(4, 3, 1), (4, 3, 2), (5, 4, 3), (3, 7, 2)])
def test_state_form_matches_factor_form_varlen(oracle_lib, m, b, T):
    N = m * b - 1
    q, k, v = _qkv(4, 2, N, 6, seed=60 + T)
    lens = np.array([N, 0, b - 2, 2 * b + 1])
    o_c = oracle.monarch_attention_varlen(q, k, v, lens, m, b, T)
    o_n = nv.monarch_attention_varlen(q, k, v, lens, m, b, T)
    np.testing.assert_allclose(o_c, o_n, rtol=0, atol=1e-13)


def test_full_lengths_give_the_unpadded_call(oracle_lib):
    q, k, v = _qkv(2, 3, 22, 8, seed=70)
    o = oracle.monarch_attention_varlen(q, k, v, np.array([22, 22]), 5, 5, 2)
    np.testing.assert_array_equal(o, oracle.monarch_attention(q, k, v, 5, 5, 2))


def test_rows_beyond_the_length_are_not_read(oracle_lib):
    q, k, v = _qkv(2, 2, 20, 8, seed=80)
    lens = np.array([7, 13])
    o1 = oracle.monarch_attention_varlen(q, k, v, lens, 4, 5, 2)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    for bi, n in enumerate(lens):
        q2[bi, :, n:] = 3.0
        k2[bi, :, n:] = -2.0
        v2[bi, :, n:] = 9.0
    np.testing.assert_array_equal(o1, oracle.monarch_attention_varlen(q2, k2, v2, lens, 4, 5, 2))


def test_varlen_rejects_lengths_out_of_range(oracle_lib):
    q, k, v = _qkv(2, 1, 8, 4, seed=90)
    for lens in ([9, 1], [-1, 3]):
        with pytest.raises(ValueError):
            oracle.monarch_attention_varlen(q, k, v, np.array(lens), 2, 4, 1)


# ---- the gradient under batch padding (oracle/backward.py) ----

def _one(n, d, seed):
    q, k, v = si.random_qkv(1, 1, n, d, "f32", seed=seed, scale=1.5)
    do = si.random_cotangent((n, d), "f32", seed=seed)
    return (x[0, 0].astype(np.float64) for x in (q, k, v)), do.astype(np.float64)


@pytest.mark.parametrize("n,m,b,T", [(5, 4, 3, 1), (5, 4, 3, 2), (2, 3, 4, 2), (7, 4, 3, 3)])
def test_padded_torch_forward_matches_oracle(n, m, b, T):
    import torch

    import oracle.backward as bw

    (q, k, v), _ = _one(n, 6, seed=100 + n + T)
    o = bw.torch_forward(*(torch.tensor(x) for x in (q, k, v)), m, b, T, batch_padding=True).numpy()
    ref = nv.monarch_attention_varlen(q[None, None], k[None, None], v[None, None], [n], m, b, T)[0, 0, :n]
    np.testing.assert_allclose(o, ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("n,m,b,T", [(4, 3, 3, 1), (4, 3, 3, 2), (2, 3, 2, 2)])
def test_padded_autograd_matches_finite_differences(n, m, b, T):
    import torch

    import oracle.backward as bw

    (q, k, v), _ = _one(n, 3, seed=110 + n + T)
    args = [torch.tensor(x, requires_grad=True) for x in (q, k, v)]
    assert torch.autograd.gradcheck(lambda a, c, e: bw.torch_forward(a, c, e, m, b, T, batch_padding=True), args,
                                    eps=1e-6, atol=1e-7)


@pytest.mark.parametrize("T", [1, 2, 3])
def test_padded_single_key_blocks_give_the_attention_gradient(T):
    """b = 1: exact attention over the real keys, so the textbook gradient."""
    import oracle.backward as bw

    (q, k, v), do = _one(7, 4, seed=120 + T)
    got = bw.autograd_grads(q, k, v, do, 12, 1, T, batch_padding=True)
    for g, w in zip(got, bw.attention_grads(q, k, v, do)):
        np.testing.assert_allclose(g, w, rtol=0, atol=1e-12)


@pytest.mark.parametrize("n,m,b", [(5, 4, 3), (9, 5, 4), (3, 6, 4)])
def test_padded_one_step_gradient_matches_fewer_blocks(n, m, b):
    """At T = 1 the real rows are those of the problem without the empty blocks,
    as functions of the real inputs, so the gradients agree too."""
    import oracle.backward as bw

    (q, k, v), do = _one(n, 5, seed=130 + n)
    got = bw.autograd_grads(q, k, v, do, m, b, 1, batch_padding=True)
    want = bw.autograd_grads(q, k, v, do, -(-n // b), b, 1)
    for g, w in zip(got, want):
        np.testing.assert_allclose(g, w, rtol=0, atol=1e-12)


@pytest.mark.parametrize("n,m,b,T", [(5, 4, 3, 2), (1, 4, 3, 2), (9, 5, 4, 3), (13, 4, 4, 2)])
def test_padded_state_form_backward_matches_autograd(n, m, b, T):
    import oracle.backward as bw

    (q, k, v), do = _one(n, 6, seed=140 + n + T)
    got = bw.state_form_backward(q, k, v, do, m, b, T, batch_padding=True)
    want = bw.autograd_grads(q, k, v, do, m, b, T, batch_padding=True)
    for g, w in zip(got, want):
        np.testing.assert_allclose(g, w, rtol=0, atol=1e-11)


def test_padded_gradient_of_an_empty_sequence_is_empty():
    import oracle.backward as bw

    z = np.zeros((0, 4))
    for g in bw.autograd_grads(z, z, z, z, 3, 3, 2, batch_padding=True) + \
            bw.state_form_backward(z, z, z, z, 3, 3, 2, batch_padding=True):
        assert g.shape == (0, 4)
