"""Pins of the gradient references (CPU): the torch forward reproduces the
pinned oracle, autograd agrees with finite differences and, for one block,
with the textbook softmax-attention gradient, and the hand-derived reverse
sweep through the state form agrees with autograd."""
import numpy as np
import pytest
import torch

import oracle.backward as bw
import oracle.naive as nv
import synth_inputs as si


def _head(n, d, seed, scale=1.5):
    q, k, v = si.random_qkv(1, 1, n, d, "f32", seed=seed, scale=scale)
    rng = np.random.default_rng(seed)
    return q[0, 0].astype(np.float64), k[0, 0].astype(np.float64), v[0, 0].astype(np.float64), rng.standard_normal((n, d))


@pytest.mark.parametrize("n,m,b,T", [(12, 3, 4, 1), (12, 3, 4, 3), (10, 3, 4, 2), (20, 4, 5, 2)])
def test_torch_forward_matches_oracle(n, m, b, T):
    q, k, v, _ = _head(n, 6, seed=n + T)
    o = bw.torch_forward(*(torch.tensor(x) for x in (q, k, v)), m, b, T).numpy()
    assert np.abs(o - nv.monarch_attention_head(q, k, v, m, b, T)).max() < 1e-12


@pytest.mark.parametrize("n,m,b,T", [(6, 2, 3, 1), (6, 2, 3, 2), (5, 2, 3, 2)])
def test_autograd_matches_finite_differences(n, m, b, T):
    q, k, v, _ = _head(n, 3, seed=10 + n + T)
    args = [torch.tensor(x, requires_grad=True) for x in (q, k, v)]
    assert torch.autograd.gradcheck(lambda a, c, e: bw.torch_forward(a, c, e, m, b, T), args, eps=1e-6, atol=1e-7)


@pytest.mark.parametrize("n,b,T", [(8, 8, 1), (8, 8, 3), (5, 8, 2)])
def test_one_block_gradient_is_softmax_attention_gradient(n, b, T):
    """m = 1: M is exact softmax attention, so are its gradients (textbook form)."""
    q, k, v, do = _head(n, 4, seed=20 + n)
    got = bw.autograd_grads(q, k, v, do, 1, b, T)
    want = bw.attention_grads(q, k, v, do)
    for g, w in zip(got, want):
        assert np.abs(g - w).max() < 1e-12


@pytest.mark.parametrize("n,m,b,d,T", [(12, 3, 4, 5, 1), (12, 3, 4, 5, 2), (12, 3, 4, 5, 3), (10, 3, 4, 6, 2),
                                       (30, 5, 6, 4, 3), (16, 2, 8, 8, 2)])
def test_state_form_backward_matches_autograd(n, m, b, d, T):
    q, k, v, do = _head(n, d, seed=30 + n + T)
    got = bw.state_form_backward(q, k, v, do, m, b, T)
    want = bw.autograd_grads(q, k, v, do, m, b, T)
    for g, w in zip(got, want):
        assert np.abs(g - w).max() < 1e-10 * max(1.0, np.abs(w).max())
