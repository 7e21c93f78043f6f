"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each check uses a worked
example or table printed in the paper, a closed form, an invariant the
construction guarantees, a special case that reduces to exact softmax
attention, or brute force on a tiny input.
"""
import os

import numpy as np
import pytest

import oracle
import oracle.naive as nv
import synth_inputs as si

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _head(m, b, d, seed=0, scale=1.5):
    q, k, v = si.random_qkv(1, 1, m * b, d, "f32", seed=seed, scale=scale)
    return q[0, 0].astype(np.float64), k[0, 0].astype(np.float64), v[0, 0].astype(np.float64)


# -- the permutation P and the index layout -------------------------------------------

def test_permutation_worked_example(oracle_lib):
    """Appendix "Monarch Background": N=6, b=3, m=2 maps (1..6) to (1,4,2,5,3,6)."""
    rows = [r for r in open(os.path.join(GOLDEN, "permutation_n6_b3_m2.txt")) if not r.startswith("#")]
    x = np.array(rows[0].split(), dtype=float)
    px = np.array(rows[1].split(), dtype=float)
    P = np.array([r.split() for r in rows[2:8]], dtype=float)
    m, b = 2, 3
    assert np.array_equal(nv.perm_matrix(m, b), P)
    assert np.array_equal(np.array([x[nv.sigma(i, m, b)] for i in range(6)]), px)
    # Qbar[j, l] = Q[l*b + j] lists the rows of P Q in order.
    qb = nv.qbar(x[:, None], m, b).reshape(-1)
    assert np.array_equal(qb, px)


def test_within_block_key_permutation_invariance(oracle_lib):
    """Permuting K and V rows jointly inside one key block leaves O unchanged:
    every quantity sums over i within a block."""
    m, b, d = 4, 6, 8
    q, k, v = _head(m, b, d, seed=3)
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], m, b, 2)
    perm = np.arange(m * b)
    rng = np.random.default_rng(0)
    for blk in range(m):
        perm[blk * b:(blk + 1) * b] = blk * b + rng.permutation(b)
    o2 = oracle.monarch_attention(q[None, None], k[perm][None, None], v[perm][None, None], m, b, 2)
    assert oracle.rel_frobenius(o2, o) < 1e-13


def test_key_block_permutation_changes_output(oracle_lib):
    """Swapping whole key blocks is NOT a symmetry: L^(0) = I pairs query block l
    with key block l.  A transposed block index in the oracle would miss this."""
    m, b, d = 4, 6, 8
    q, k, v = _head(m, b, d, seed=4)
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], m, b, 1)
    perm = np.concatenate([np.arange(b, 2 * b), np.arange(0, b), np.arange(2 * b, m * b)])
    o2 = oracle.monarch_attention(q[None, None], k[perm][None, None], v[perm][None, None], m, b, 1)
    assert oracle.rel_frobenius(o2, o) > 1e-3


def test_residue_classes_are_independent(oracle_lib):
    """Query rows of one residue class j (rows l*b + j) feed only the output
    rows of that class: every chain alpha_R[:, j] -> R[:, j] -> alpha_L[j] -> L[j]
    stays inside class j."""
    m, b, d = 5, 4, 8
    q, k, v = _head(m, b, d, seed=5)
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], m, b, 3)[0, 0]
    j0 = 2
    q2 = q.copy()
    q2[j0::b] += 0.75
    o2 = oracle.monarch_attention(q2[None, None], k[None, None], v[None, None], m, b, 3)[0, 0]
    other = np.array([r % b != j0 for r in range(m * b)])
    assert np.array_equal(o2[other], o[other])
    assert np.abs(o2[~other] - o[~other]).max() > 1e-6


# -- Monarch structure ----------------------------------------------------------------

@pytest.mark.parametrize("m,b,T", [(3, 4, 1), (4, 3, 2), (5, 5, 3)])
def test_dense_monarch_forms_agree_and_apply(oracle_lib, m, b, T):
    """Entrywise form (eq. monarch_entrywise) == P^T blockdiag(L_j^T) P blockdiag(R_k)
    (Sec. 2), and M V equals the structured output of eq. monarch_multiply."""
    d = 6
    q, k, v = _head(m, b, d, seed=10 + T)
    L, R = nv.factors(q, k, m, b, T)
    M1 = nv.dense_monarch(L, R)
    M2 = nv.dense_monarch_factored(L, R)
    assert np.abs(M1 - M2).max() < 1e-14
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], m, b, T)[0, 0]
    assert oracle.rel_frobenius(o, M1 @ v) < 1e-13


@pytest.mark.parametrize("m,b,T", [(3, 4, 1), (4, 3, 3)])
def test_monarch_is_row_stochastic(m, b, T):
    """L[j,:,l] and R[k,j,:] on the simplex imply M >= 0 with unit row sums (Sec. 3)."""
    q, k, v = _head(m, b, 5, seed=20 + T)
    L, R = nv.factors(q, k, m, b, T)
    assert (L >= 0).all() and (R >= 0).all()
    assert np.allclose(L.sum(axis=1), 1.0, atol=1e-14)   # over k
    assert np.allclose(R.sum(axis=2), 1.0, atol=1e-14)   # over i
    M = nv.dense_monarch(L, R)
    assert (M >= 0).all()
    assert np.allclose(M.sum(axis=1), 1.0, atol=1e-13)


# -- the variational form of softmax ---------------------------------------------------

def test_variational_identity_closed_form():
    """softmax(z) attains <p, z> + H(p) = logsumexp(z) (eq. softmax_variational, App. A)."""
    rng = np.random.default_rng(1)
    for n in (2, 5, 17):
        z = 3.0 * rng.standard_normal(n)
        p = np.exp(z - z.max())
        p /= p.sum()
        val = p @ z - np.sum(p * np.log(p))
        assert abs(val - nv.log_sum_exp(z)) < 1e-12


def test_variational_identity_brute_force_simplex():
    """On a 401-point-per-axis grid of the 3-simplex no point beats softmax(z)."""
    z = np.array([0.3, -1.1, 0.8])
    n = 400
    a1, a2 = np.meshgrid(np.arange(n + 1), np.arange(n + 1), indexing="ij")
    keep = a1 + a2 <= n
    p = np.stack([a1[keep], a2[keep], n - a1[keep] - a2[keep]], axis=1) / n
    with np.errstate(divide="ignore", invalid="ignore"):
        ent = -np.where(p > 0, p * np.log(p), 0.0).sum(axis=1)
    vals = p @ z + ent
    lse = nv.log_sum_exp(z)
    assert vals.max() <= lse + 1e-12
    assert vals.max() > lse - 1e-4


@pytest.mark.parametrize("m,b", [(3, 4), (4, 4)])
def test_separable_objective_matches_dense(m, b):
    """f(M) from the factors with the separable entropy (Sec. 3, Softmax Objective)
    equals f evaluated on the dense Monarch matrix."""
    q, k, v = _head(m, b, 6, seed=30)
    L, R = nv.factors(q, k, m, b, 2)
    assert abs(nv.objective_monarch(L, R, q, k) - nv.objective_dense(nv.dense_monarch(L, R), q, k)) < 1e-10


def _perturb_simplex(p, rng, eps):
    w = rng.dirichlet(np.ones(len(p)))
    return (1 - eps) * p + eps * w


@pytest.mark.parametrize("T", [1, 2, 3])
def test_updates_are_block_maximisers(T):
    """Each half-step is the exact maximiser of f over its factor with the other
    fixed (App. "Updates"): no simplex perturbation of one R row or one L column
    increases f, evaluated densely from eq. softmax_variational_attention."""
    m, b, d = 3, 4, 5
    q, k, v = _head(m, b, d, seed=40 + T, scale=2.0)
    L, R, hist = nv.factors(q, k, m, b, T, history=True)
    rng = np.random.default_rng(T)
    # the last R update (L fixed at the previous L) and the last L update
    L_prev, R_last = hist[-2]
    f_r = nv.objective_dense(nv.dense_monarch(L_prev, R_last), q, k)
    f_l = nv.objective_dense(nv.dense_monarch(L, R), q, k)
    for _ in range(40):
        kk, j = rng.integers(m), rng.integers(b)
        R2 = R_last.copy()
        R2[kk, j] = _perturb_simplex(R2[kk, j], rng, rng.choice([1e-3, 1e-2, 0.3]))
        assert nv.objective_dense(nv.dense_monarch(L_prev, R2), q, k) <= f_r + 1e-12
        j, l = rng.integers(b), rng.integers(m)
        L2 = L.copy()
        L2[j, :, l] = _perturb_simplex(L2[j, :, l], rng, rng.choice([1e-3, 1e-2, 0.3]))
        assert nv.objective_dense(nv.dense_monarch(L2, R), q, k) <= f_l + 1e-12


@pytest.mark.parametrize("m,b", [(3, 4), (4, 2), (2, 5)])
def test_ascent_and_upper_bound(m, b):
    """f(M) never decreases over the half-steps and never exceeds f at exact
    softmax, sum over rows of logsumexp(s q K^T) (App. A applied row-wise)."""
    q, k, v = _head(m, b, 6, seed=50 + m, scale=2.0)
    _, _, hist = nv.factors(q, k, m, b, 4, history=True)
    vals = [nv.objective_dense(nv.dense_monarch(Lh, Rh), q, k) for Lh, Rh in hist[1:]]
    assert all(b2 >= a2 - 1e-12 for a2, b2 in zip(vals, vals[1:]))
    s = 1.0 / np.sqrt(q.shape[1])
    bound = sum(nv.log_sum_exp(s * q[r] @ k.T) for r in range(m * b))
    assert vals[-1] <= bound + 1e-12


# -- special cases with a textbook answer -----------------------------------------------

@pytest.mark.parametrize("m,b,T", [(1, 12, 1), (1, 12, 3), (12, 1, 1), (12, 1, 2)])
def test_single_block_is_exact_softmax_attention(oracle_lib, m, b, T):
    """m = 1 (one block: L = 1, R = row softmax) or b = 1 (R = 1, L = row
    softmax) makes M exactly softmax(s Q K^T) for every T."""
    q, k, v = _head(m, b, 8, seed=60)
    ref = nv.dense_softmax_attention(q, k, v)
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], m, b, T)[0, 0]
    assert oracle.rel_frobenius(o, ref) < 1e-13
    assert oracle.rel_frobenius(nv.monarch_attention_head(q, k, v, m, b, T), ref) < 1e-13


@pytest.mark.parametrize("m,b,T", [(4, 5, 1), (6, 3, 3)])
def test_identical_queries_give_exact_attention(oracle_lib, m, b, T):
    """With all query rows equal, L[j,k,l] becomes the softmax over k of the
    block log-sum-exps and M equals softmax attention for every T >= 1."""
    q, k, v = _head(m, b, 8, seed=70)
    q[:] = q[0]
    ref = nv.dense_softmax_attention(q, k, v)
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], m, b, T)[0, 0]
    assert oracle.rel_frobenius(o, ref) < 1e-13


def test_zero_keys_give_mean_of_values(oracle_lib):
    """K = 0: R uniform over i, c_L = -log b, L uniform over k, so M = 1/N."""
    m, b, d = 4, 5, 8
    q, k, v = _head(m, b, d, seed=80)
    k[:] = 0.0
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], m, b, 2)[0, 0]
    assert np.abs(o - v.mean(axis=0)).max() < 1e-14


# -- the two formulations and the work count -------------------------------------------------

@pytest.mark.parametrize("m,b,d,T", [(2, 3, 4, 1), (5, 3, 7, 2), (3, 7, 16, 3), (8, 8, 16, 2), (4, 9, 5, 4)])
def test_state_form_matches_factor_form(oracle_lib, m, b, d, T):
    """The C state form (alpha/c only) equals the materialised-factor form."""
    q, k, v = si.random_qkv(2, 1, m * b, d, "bf16", seed=m * 100 + b, scale=2.0)
    o1 = oracle.monarch_attention(q, k, v, m, b, T)
    o2 = nv.monarch_attention(q, k, v, m, b, T)
    assert oracle.rel_frobenius(o1, o2) < 1e-12


def test_macs_reproduce_paper_flop_tables():
    """T(2Nbd + 2Nmd) + Nbd multiply-adds per head reproduces every MonarchAttention
    entry of the BART table and tab:dit, and 2 N^2 d the softmax entries."""
    rows = [r.split() for r in open(os.path.join(GOLDEN, "attention_flop_tables.txt")) if not r.startswith("#")]
    for src, heads, N, d, b, T, ma, sm in rows:
        heads, N, d, b, T = map(int, (heads, N, d, b, T))
        m = N // b
        got = heads * oracle.macs_per_head(N, m, b, d, T) / 1e9
        assert abs(got - float(ma)) / float(ma) < 0.01, (src, N, got, ma)
        soft = heads * 2 * N * N * d / 1e9
        assert abs(soft - float(sm)) / float(sm) < 0.01, (src, N, soft, sm)
    (hm, hs, N, d, b, T, tot), = [r.split() for r in open(os.path.join(GOLDEN, "dit_half_layers.txt"))
                                  if not r.startswith("#")]
    hm, hs, N, d, b, T = map(int, (hm, hs, N, d, b, T))
    got = (hm * oracle.macs_per_head(N, N // b, b, d, T) + hs * 2 * N * N * d) / 1e9
    assert abs(got - float(tot)) / float(tot) < 0.01


def test_dense_attention_rows(oracle_lib):
    """The C exact-attention helper agrees with the numpy definition."""
    q, k, v = si.random_qkv(1, 2, 40, 8, "f32", seed=9, scale=1.5)
    rows = np.array([0, 7, 39])
    got = oracle.dense_attention_rows(q, k, v, rows)
    for h in range(2):
        ref = nv.dense_softmax_attention(q[0, h], k[0, h], v[0, h])[rows]
        assert np.abs(got[0, h] - ref).max() < 1e-13


# -- sequence lengths that are not a multiple of b (Appendix "Padding and Masking") ------

def _padded_head(n, m, b, d, seed):
    q, k, v = _head(m, b, d, seed=seed)
    return q[:n], k[:n], v[:n]


@pytest.mark.parametrize("n,m,b", [(10, 3, 4), (197, 15, 14), (7, 2, 4)])
def test_padding_zeroes_the_padded_columns_of_M(n, m, b):
    """The mask omega (-inf on Z_R at key positions >= N) makes the last
    m*b - N columns of the padded Monarch matrix exactly zero, which is what
    the appendix asks of it; the rows still sum to one."""
    q, k, v = _padded_head(n, m, b, 6, seed=90 + n)
    L, R = nv.factors(q, k, m, b, 2)
    M = nv.dense_monarch(L, R)
    assert np.all(M[:, n:] == 0.0)
    assert np.all(M >= 0) and np.allclose(M.sum(axis=1), 1.0, atol=1e-12)
    # and O is M V on the real rows
    assert np.abs(nv.monarch_apply(L, R, v) - M[:n, :n] @ v).max() < 1e-12


def test_padding_ignores_padded_key_and_value_rows():
    """Whatever the padded K and V rows hold, the real outputs are the same
    (their R entries are exactly zero)."""
    n, m, b, d = 10, 3, 4, 6
    q, k, v = _padded_head(n, m, b, d, seed=95)
    ref = nv.monarch_attention_head(q, k, v, m, b, 2)
    rng = np.random.default_rng(5)
    qp, kp, vp = (nv.pad_rows(x, m, b) for x in (q, k, v))
    kp[n:] = 4 * rng.normal(size=(m * b - n, d))
    vp[n:] = 4 * rng.normal(size=(m * b - n, d))
    L, R = nv.factors(qp, kp, m, b, 2, n=n)
    got = nv.monarch_apply(L, R, vp)[:n]
    assert np.abs(got - ref).max() < 1e-13


def test_padded_query_rows_take_part():
    """Padded query rows are rows of the padded problem: they shape alpha_R and
    c_R, so their values change the real outputs.  (This is why the pad value
    is a convention; zero rows are the one used everywhere here.)"""
    n, m, b, d = 10, 3, 4, 6
    q, k, v = _padded_head(n, m, b, d, seed=96)
    ref = nv.monarch_attention_head(q, k, v, m, b, 2)
    qp, kp, vp = (nv.pad_rows(x, m, b) for x in (q, k, v))
    qp[n:] = 3.0
    L, R = nv.factors(qp, kp, m, b, 2, n=n)
    assert np.abs(nv.monarch_apply(L, R, vp)[:n] - ref).max() > 1e-6


@pytest.mark.parametrize("n,b,T", [(5, 8, 1), (11, 16, 3), (1, 4, 2)])
def test_single_padded_block_is_exact_attention(oracle_lib, n, b, T):
    """m = 1 with N < b: one block whose padded keys are masked, so M is the
    exact softmax attention of the N real tokens."""
    q, k, v = _padded_head(n, 1, b, 8, seed=97 + n)
    ref = nv.dense_softmax_attention(q, k, v)
    o = oracle.monarch_attention(q[None, None], k[None, None], v[None, None], 1, b, T)[0, 0]
    assert o.shape == (n, 8)
    assert oracle.rel_frobenius(o, ref) < 1e-13
    assert oracle.rel_frobenius(nv.monarch_attention_head(q, k, v, 1, b, T), ref) < 1e-13


@pytest.mark.parametrize("n,m,b,T", [(10, 3, 4, 1), (197, 15, 14, 2), (33, 3, 16, 3), (61, 4, 16, 2), (130, 2, 128, 2)])
def test_state_form_matches_factor_form_padded(oracle_lib, n, m, b, T):
    """The C state form with its internal padding equals the materialised-factor form."""
    q, k, v = si.random_qkv(2, 1, n, 8, "bf16", seed=n * 7 + b, scale=2.0)
    o1 = oracle.monarch_attention(q, k, v, m, b, T)
    o2 = nv.monarch_attention(q, k, v, m, b, T)
    assert o1.shape == q.shape
    assert oracle.rel_frobenius(o1, o2) < 1e-12


def test_padding_rejects_m_other_than_ceil_n_over_b(oracle_lib):
    q, k, v = si.random_qkv(1, 1, 10, 4, "f32", seed=1)
    for m in (2, 4):   # ceil(10 / 4) = 3
        with pytest.raises(ValueError):
            oracle.monarch_attention(q, k, v, m, 4, 1)


# -- the objective as a convergence diagnostic ---------------------------------------------

@pytest.mark.parametrize("m,b,T", [(3, 4, 1), (4, 4, 3), (2, 5, 2)])
def test_objective_after_l_update_is_sum_of_row_logsumexps(m, b, T):
    """After each L update, f(M) (separable form of Sec. 3, and the dense form
    of eq. softmax_variational_attention) equals the sum over query rows of the
    logsumexp of the L-update logits."""
    q, k, v = _head(m, b, 6, seed=110 + T, scale=2.0)
    _, _, hist = nv.factors(q, k, m, b, T, history=True)
    for t in range(1, T + 1):
        L, R = hist[2 * t]          # (L^(t), R^(t))
        f_sep = nv.objective_monarch(L, R, q, k)
        f_dense = nv.objective_dense(nv.dense_monarch(L, R), q, k)
        f_lse = nv.objective_after_l_update(R, q, k, m, b)
        assert abs(f_sep - f_dense) < 1e-10
        assert abs(f_lse - f_sep) < 1e-10


def test_objective_padded_sum_of_row_logsumexps():
    """The same identity on a padded problem (all m*b rows, zero padding, masked keys)."""
    n, m, b = 10, 3, 4
    q, k, v = _padded_head(n, m, b, 6, seed=120)
    L, R = nv.factors(q, k, m, b, 2)
    qp, kp = nv.pad_rows(q, m, b), nv.pad_rows(k, m, b)
    assert abs(nv.objective_after_l_update(R, q, k, m, b) - nv.objective_monarch(L, R, qp, kp)) < 1e-10


@pytest.mark.parametrize("m,b,T", [(3, 4, 3), (5, 3, 2), (4, 9, 4)])
def test_c_objective_matches_separable_form(oracle_lib, m, b, T):
    """The C oracle's per-step objective (separable form from its states) equals
    the numpy separable form on the materialised factors."""
    q, k, v = _head(m, b, 7, seed=130 + m, scale=2.0)
    _, f = oracle.monarch_attention_objective(q[None, None], k[None, None], v[None, None], m, b, T)
    _, _, hist = nv.factors(q, k, m, b, T, history=True)
    ref = [nv.objective_monarch(*hist[2 * t], q, k) for t in range(1, T + 1)]
    assert np.abs(f[0, 0] - ref).max() < 1e-9 * max(1.0, np.abs(ref).max())
    assert all(b2 >= a2 - 1e-12 for a2, b2 in zip(f[0, 0], f[0, 0][1:]))   # ascent over the steps
