"""The per-unit error measures of the GPU parity tests find an error planted
in one residue class (query rows l*b + j) or one key block (rows k*b + i),
including with a ragged last block (CPU only)."""
import numpy as np

import parity


def _ref(shape, seed=0):
    return np.random.RandomState(seed).standard_normal(shape)


def test_class_errors_find_one_class():
    B, H, m, b, d = 2, 3, 5, 7, 8
    ref = _ref((B, H, m * b - 3, d))
    o = ref.copy()
    o[1, 2, 4::b] *= 1.2  # class j = 4 of (batch 1, head 2): rows 4, 11, 18, 25
    err, where = parity.worst_class(o, ref, b)
    assert where == (1, 2, 4)
    np.testing.assert_allclose(err, 0.2, rtol=1e-12)
    rel = parity.class_errors(o, ref, b)
    assert np.count_nonzero(rel) == 1


def test_block_errors_find_one_block():
    B, H, m, b, d = 1, 2, 6, 5, 4
    ref = _ref((B, H, m * b - 2, d), seed=1)
    o = ref.copy()
    o[0, 1, 3 * b:4 * b] -= 0.5 * ref[0, 1, 3 * b:4 * b]  # key block k = 3 of head 1
    rel = parity.block_errors(o, ref, b)
    assert rel.shape == (B, H, m)
    assert np.unravel_index(int(np.argmax(rel)), rel.shape) == (0, 1, 3)
    np.testing.assert_allclose(rel.max(), 0.5, rtol=1e-12)
    assert np.count_nonzero(rel) == 1


def test_ragged_last_block_and_zero_rows():
    b = 4
    ref = _ref((1, 1, 10, 3), seed=2)  # blocks of 4, 4 and 2 rows
    ref[0, 0, 8:] = 0.0               # the ragged block is all zero in the reference
    o = ref.copy()
    assert parity.block_errors(o, ref, b)[0, 0, 2] == 0.0
    o[0, 0, 9, 1] = 1e-3              # a nonzero where the reference is zero
    assert np.isinf(parity.block_errors(o, ref, b)[0, 0, 2])


def test_worst_grad_unit_names_the_gradient():
    m, b, d = 4, 4, 3
    shape = (1, 1, m * b, d)
    rq, rk, rv = _ref(shape, 3), _ref(shape, 4), _ref(shape, 5)
    dq, dk, dv = rq.copy(), rk.copy(), rv.copy()
    dv[0, 0, 2 * b:3 * b] *= 1.1      # key block 2 of dV
    dq[0, 0, 1::b] *= 1.05            # residue class 1 of dQ
    err, name, where = parity.worst_grad_unit(dq, dk, dv, rq, rk, rv, b)
    assert (name, where) == ("dv", (0, 0, 2))
    np.testing.assert_allclose(err, 0.1, rtol=1e-12)
    assert parity.class_bar(2e-2) == 4e-2
