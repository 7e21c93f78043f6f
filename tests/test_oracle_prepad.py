"""Pins of the oracle's pre-padding (Appendix "Padding and Masking", its last
sentence: the padding rows come first, and the key mask then removes the
positions below N' - N instead of those from N on).

* The C oracle equals the numpy one (different code: explicit factors,
  per-(k, j) and per-(j, l) loops).
* Relabelling: the map x -> N' - 1 - x of the m*b positions sends block l to
  m - 1 - l and row j to b - 1 - j.  It keeps L^(0) = I (it pairs block l
  with key block l on both sides), it permutes the keys within a block (the
  R softmax) and the key blocks (the L softmax), and it turns pre-padding
  into post-padding.  So the pre-padded result is the post-padded result of
  the row-reversed inputs, row-reversed, for every T.
* One block (m = 1), and one key per block (b = 1, batch padding): exact
  softmax attention over the real keys at every T.
* M is row-stochastic with zero columns at the padded positions.
* An off-by-one in the mask and a mask on the wrong side are caught.
"""
import numpy as np
import pytest

import oracle
import oracle.naive as nv
import synth_inputs as si


def rev(x):
    return np.ascontiguousarray(x[:, :, ::-1])


SHAPES = [(2, 2, 37, 8, 5, 8, 2), (1, 3, 60, 16, 4, 16, 3), (1, 2, 64, 8, 8, 8, 1), (2, 1, 13, 4, 2, 7, 4),
          (1, 1, 1, 8, 1, 16, 2)]


@pytest.mark.parametrize("B,H,N,d,m,b,T", SHAPES)
def test_c_equals_numpy(B, H, N, d, m, b, T):
    q, k, v = si.random_qkv(B, H, N, d, "f32", seed=N + b, scale=1.5)
    a = oracle.monarch_attention_prepad(q, k, v, m, b, T)
    c = nv.monarch_attention(q, k, v, m, b, T, pre_pad=True)
    assert np.abs(a - c).max() <= 1e-12 * max(1.0, np.abs(c).max())
    lens = np.array([N, 0, 1, max(1, N // 3)][:B]) if B > 1 else np.array([max(1, N // 2)])
    a = oracle.monarch_attention_prepad(q, k, v, m, b, T, lens=lens)
    c = nv.monarch_attention_varlen(q, k, v, lens, m, b, T, pre_pad=True)
    assert np.abs(a - c).max() <= 1e-12 * max(1.0, np.abs(c).max())
    for bi, n in enumerate(lens):
        assert np.all(a[bi, :, : N - n] == 0.0)


@pytest.mark.parametrize("B,H,N,d,m,b,T", SHAPES)
def test_relabelling_turns_pre_into_post_padding(B, H, N, d, m, b, T):
    q, k, v = si.random_qkv(B, H, N, d, "f32", seed=7 * N + b, scale=1.5)
    pre = nv.monarch_attention(q, k, v, m, b, T, pre_pad=True)
    post = rev(nv.monarch_attention(rev(q), rev(k), rev(v), m, b, T))
    assert np.abs(pre - post).max() <= 1e-12 * max(1.0, np.abs(post).max())
    # the left-padded batch: its real rows are the last ones, reversed they are the first
    lens = np.array([N, 0, 1, max(1, N // 3)][:B]) if B > 1 else np.array([max(1, N // 2)])
    pre = oracle.monarch_attention_prepad(q, k, v, m, b, T, lens=lens)
    post = rev(oracle.monarch_attention_varlen(rev(q), rev(k), rev(v), lens, m, b, T))
    assert np.abs(pre - post).max() <= 1e-12 * max(1.0, np.abs(post).max())


@pytest.mark.parametrize("T", [1, 2, 3])
def test_one_block_is_exact_attention(T):
    """m = 1: the block of b >= N positions holds b - N padded keys first;
    the L factor is 1 and R is the masked softmax, i.e. exact attention."""
    N, b = 5, 16
    q, k, v = si.random_qkv(1, 2, N, 8, "f32", seed=3, scale=1.5)
    got = oracle.monarch_attention_prepad(q, k, v, 1, b, T)
    for h in range(2):
        want = nv.dense_softmax_attention(q[0, h], k[0, h], v[0, h])
        assert np.abs(got[0, h] - want).max() <= 1e-12


@pytest.mark.parametrize("T", [1, 2])
def test_one_key_per_block_is_exact_attention(T):
    """b = 1 with a left-padded batch: blocks of padding only get R = 0 and no
    L weight, the others hold one real key each: exact attention over the
    real keys."""
    N, m = 9, 9
    q, k, v = si.random_qkv(2, 1, N, 8, "f32", seed=4, scale=1.5)
    lens = np.array([9, 4])
    got = oracle.monarch_attention_prepad(q, k, v, m, 1, T, lens=lens)
    for bi, n in enumerate(lens):
        want = nv.dense_softmax_attention(q[bi, 0, N - n:], k[bi, 0, N - n:], v[bi, 0, N - n:])
        assert np.abs(got[bi, 0, N - n:] - want).max() <= 1e-12
        assert np.all(got[bi, 0, : N - n] == 0.0)


def test_monarch_matrix_has_zero_columns_at_the_front_padding():
    N, m, b, T = 13, 3, 5, 2
    q, k, _ = si.random_qkv(1, 1, N, 8, "f32", seed=5, scale=1.5)
    L, R = nv.factors(q[0, 0], k[0, 0], m, b, T, pre_pad=True)
    M = nv.dense_monarch(L, R)
    P = m * b - N
    assert np.all(M >= 0.0)
    assert np.allclose(M.sum(axis=1), 1.0, atol=1e-12)
    assert np.all(M[:, :P] == 0.0)
    assert np.all(M[:, P:].sum(axis=0) > 0.0)


def _mask_off_by_one(n, m, b, pre=False):
    om = np.zeros((m, b))
    for kk in range(m):
        for i in range(b):
            pos = kk * b + i
            real = pos > m * b - n if pre else pos < n     # one real key lost at the front
            if not real:
                om[kk, i] = -np.inf
    return om


def _mask_wrong_side(n, m, b, pre=False):
    om = np.zeros((m, b))
    for kk in range(m):
        for i in range(b):
            if kk * b + i >= n:                            # the post-padding mask with pre-padded rows
                om[kk, i] = -np.inf
    return om


@pytest.mark.parametrize("mutant", [_mask_off_by_one, _mask_wrong_side])
def test_mask_mutants_are_caught(monkeypatch, mutant):
    monkeypatch.setattr(nv, "key_mask", mutant)
    N, b = 5, 16
    q, k, v = si.random_qkv(1, 1, N, 8, "f32", seed=3, scale=1.5)
    got = nv.monarch_attention(q, k, v, 1, b, 2, pre_pad=True)
    want = nv.dense_softmax_attention(q[0, 0], k[0, 0], v[0, 0])
    assert not np.allclose(got[0, 0], want, atol=1e-6)
