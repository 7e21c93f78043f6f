"""Materialised-factor fp64 oracle of MonarchAttention (numpy).

TEST INFRASTRUCTURE ONLY: used by the test suite to pin the C oracle; the
product path never imports it.

This is the direct form of the alternating maximisation (Sec. 3, "Alternating
Maximization with Constraints", eqs. R_update, L_update, beta_r, beta_l), with
the factors L[j, k, l] and R[k, j, i] held explicitly, followed by the Monarch
product of eq. monarch_multiply.  It is written with small per-(k, j) and
per-(j, l) vector operations so that each line can be checked against one
equation; it is meant for small N only.

Indices are 0-based: query row (l, j) is row l*b + j of Q and key row (k, i)
is row k*b + i of K (the rows of Qbar and Kbar in eq. beta_r).  Q is scaled by
s = 1/sqrt(d) before use (Sec. 2, attention footnote).

A length N that is not a multiple of b follows Appendix "Padding and
Masking": m = ceil(N / b), Q, K, V post-padded to m*b rows (zero rows unless
the caller passes padded arrays), the mask omega (-inf at key positions
k*b + i >= N) added to Z_R before the softmax of eq. R_update, and the first
N rows of O kept.

The same appendix covers a batch of sequences padded to a common length.
There m and b are fixed for the batch, so a shorter sequence can have whole
key blocks of padding, whose row of omega is -inf throughout and whose
softmax the paper leaves undefined.  The reading taken here
(``batch_padding=True``): such a block gets R = 0, and the L update leaves
it out (Z_L = -inf for it), so that M keeps unit row sums with zero columns
at every padded key.  A sequence of length 0 has M = 0.
"""
from __future__ import annotations

import numpy as np


def sigma(i: int, m: int, b: int) -> int:
    """Index map of the "transpose" permutation P (Sec. 2): (P x)_i = x_sigma(i)."""
    return b * (i % m) + i // m


def perm_matrix(m: int, b: int) -> np.ndarray:
    """P as an N x N 0/1 matrix whose row i is e_sigma(i)."""
    n = m * b
    p = np.zeros((n, n))
    for i in range(n):
        p[i, sigma(i, m, b)] = 1.0
    return p


def qbar(q: np.ndarray, m: int, b: int) -> np.ndarray:
    """Qbar[j, l] = Q[l*b + j] (rows of P Q grouped in b blocks of m)."""
    n, d = q.shape
    out = np.empty((b, m, d))
    for j in range(b):
        for l in range(m):
            out[j, l] = q[l * b + j]
    return out


def kbar(k: np.ndarray, m: int, b: int) -> np.ndarray:
    """Kbar[k, i] = K[k*b + i] (consecutive blocks of b rows)."""
    n, d = k.shape
    out = np.empty((m, b, d))
    for kk in range(m):
        for i in range(b):
            out[kk, i] = k[kk * b + i]
    return out


def pad_rows(x: np.ndarray, m: int, b: int) -> np.ndarray:
    """Post-pad the rows of x with zero rows to m*b rows."""
    out = np.zeros((m * b,) + x.shape[1:])
    out[: x.shape[0]] = x
    return out


def key_mask(n: int, m: int, b: int, pre: bool = False) -> np.ndarray:
    """omega[k, i] = 0 at real key positions and -inf at padded ones (Appendix
    "Padding and Masking").  Post-padding: position k*b + i is real when it is
    below n.  Pre-padding: the m*b - n padded rows come first, so a position
    is real when it is at least m*b - n (the appendix's condition with
    0-based positions)."""
    omega = np.zeros((m, b))
    for k in range(m):
        for i in range(b):
            pos = k * b + i
            real = pos >= m * b - n if pre else pos < n
            if not real:
                omega[k, i] = -np.inf
    return omega


def front_pad_rows(x: np.ndarray, m: int, b: int) -> np.ndarray:
    """Pre-pad the rows of x with zero rows to m*b rows (real rows last)."""
    out = np.zeros((m * b,) + x.shape[1:])
    out[m * b - x.shape[0]:] = x
    return out


def live_blocks(n: int, b: int) -> int:
    """Key blocks that hold at least one real key, ceil(n / b)."""
    return -(-n // b)


def _softmax(z: np.ndarray) -> np.ndarray:
    e = np.exp(z - z.max())
    return e / e.sum()


def _xlogx_sum(p: np.ndarray) -> float:
    nz = p > 0
    return float(np.sum(p[nz] * np.log(p[nz])))


def r_update(L: np.ndarray, Qb: np.ndarray, Kb: np.ndarray, omega=None) -> np.ndarray:
    """R = softmax_i(beta_R / c_R + omega) with beta_R, c_R from L (eqs. R_update, beta_r);
    omega is the padding mask, absent when N = m*b."""
    b, m, _ = L.shape
    R = np.empty((m, b, b))
    for k in range(m):
        for j in range(b):
            if omega is not None and np.all(np.isneginf(omega[k])):
                R[k, j] = 0.0                     # no real key in block k (batch padding)
                continue
            alpha_r = L[j, k, :] @ Qb[j]          # sum_l L[j,k,l] Qbar[j,l,:]
            c_r = L[j, k, :].sum()                # sum_l L[j,k,l]
            beta_r = Kb[k] @ alpha_r              # beta_R[k,j,i] = <alpha_R[k,j], Kbar[k,i]>
            z_r = beta_r / c_r
            if omega is not None:
                z_r = z_r + omega[k]
            R[k, j] = _softmax(z_r)
    return R


def l_update(R: np.ndarray, Qb: np.ndarray, Kb: np.ndarray, live=None) -> np.ndarray:
    """L = softmax_k(beta_L - c_L) with beta_L, c_L from R (eqs. L_update, beta_l).
    live: the key blocks that hold a real key, as a count (blocks k < live,
    post-padding) or a boolean array over k; the others (batch padding) get
    Z_L = -inf, and L = 0 when no block does."""
    m, b, _ = R.shape
    if live is None:
        live = m
    mask = np.arange(m) < live if np.isscalar(live) else np.asarray(live, dtype=bool)
    L = np.zeros((b, m, m))
    if not mask.any():
        return L
    for j in range(b):
        alpha_l = np.stack([R[k, j] @ Kb[k] for k in range(m)])       # [k, v]
        c_l = np.array([_xlogx_sum(R[k, j]) for k in range(m)])        # sum_i R log R
        for l in range(m):
            beta_l = alpha_l @ Qb[j, l]                                 # over k
            L[j, mask, l] = _softmax((beta_l - c_l)[mask])
    return L


def _f64(*xs):
    return [np.asarray(x, dtype=np.float64) for x in xs]


def monarch_apply(L: np.ndarray, R: np.ndarray, v: np.ndarray, pre_pad: bool = False) -> np.ndarray:
    """O = M V by the two-step product of eq. monarch_multiply; v with N <= m*b rows
    (zero-padded after them, or before them with pre_pad), O with the same N rows."""
    (v,) = _f64(v)
    b, m, _ = L.shape
    n = v.shape[0]
    if n < m * b:
        v = front_pad_rows(v, m, b) if pre_pad else pad_rows(v, m, b)
    Vb = kbar(v, m, b)
    Y = np.empty((b, m, v.shape[1]))
    for j in range(b):
        for k in range(m):
            Y[j, k] = R[k, j] @ Vb[k]            # sum_i R[k,j,i] Vbar[k,i,:]
    O = np.empty_like(v)
    for l in range(m):
        for j in range(b):
            O[l * b + j] = L[j, :, l] @ Y[j]     # sum_k L[j,k,l] Y[j,k,:]
    return O[m * b - n:] if pre_pad else O[:n]


def factors(q, k, m, b, T, *, history=False, n=None, batch_padding=False, pre_pad=False):
    """Run T (R, L) update pairs from L^(0) = I (Sec. 3).  q, k: one head [N, d].

    N < m*b rows are zero-padded to m*b, after the real rows or, with
    pre_pad, before them.  Arrays that already have m*b rows with n < m*b
    are taken as padded by the caller (post-padding only: rows >= n are
    padding, whatever they hold).  With batch_padding, n may be any length
    0..m*b (whole blocks of padding allowed, see the module docstring);
    otherwise m = ceil(n / b).  Returns (L, R) after T steps; with
    history=True also the list of (L, R) pairs after every half-step,
    starting with (L^(0), None).
    """
    q, k = _f64(q, k)
    rows, d = q.shape
    n = rows if n is None else n
    if batch_padding:
        assert 0 <= n <= m * b and T >= 1
    else:
        assert (m - 1) * b < n <= m * b and T >= 1    # m = ceil(N / b)
    if rows < m * b:
        assert rows == n
        pad = front_pad_rows if pre_pad else pad_rows
        q, k = pad(q, m, b), pad(k, m, b)
    assert q.shape[0] == m * b and (not pre_pad or rows == n)
    omega = key_mask(n, m, b, pre=pre_pad) if n < m * b else None
    # key blocks holding a real key: the first ceil(n / b), or with pre-padding the last ones
    live = live_blocks(n, b) if omega is None or not pre_pad else ~np.all(np.isneginf(omega), axis=1)
    s = 1.0 / np.sqrt(d)
    Qb = qbar(s * q, m, b)
    Kb = kbar(k, m, b)
    L = np.stack([np.eye(m) for _ in range(b)])    # L^(0)[j,k,l] = delta_kl
    R = None
    hist = [(L, None)]
    for _ in range(T):
        R = r_update(L, Qb, Kb, omega)              # R before L in every step
        hist.append((L, R))
        L = l_update(R, Qb, Kb, live)
        hist.append((L, R))
    return (L, R, hist) if history else (L, R)


def monarch_attention_head(q, k, v, m, b, T, pre_pad=False):
    """One head: O = M^(T) V.  q, k, v: [N, d] (widened to float64); with
    pre_pad the N rows are pre-padded to m*b instead of post-padded."""
    L, R = factors(q, k, m, b, T, pre_pad=pre_pad)
    return monarch_apply(L, R, v, pre_pad=pre_pad)


def monarch_attention(q, k, v, m, b, T, pre_pad=False):
    """All heads: q, k, v [B, H, N, d] (widened to float64)."""
    q, k, v = _f64(q, k, v)
    out = np.empty_like(v)
    for bi in range(q.shape[0]):
        for h in range(q.shape[1]):
            out[bi, h] = monarch_attention_head(q[bi, h], k[bi, h], v[bi, h], m, b, T, pre_pad=pre_pad)
    return out


def monarch_attention_varlen(q, k, v, lens, m, b, T, pre_pad=False):
    """A batch of padded sequences: q, k, v [B, H, N, d], lens[B] <= N real rows
    per batch element.  Post-padding: the real rows are the first lens[beta]
    rows, each head is the single-sequence problem of those rows post-padded
    to m*b at the batch's m and b (with ``batch_padding``), and rows
    >= lens[beta] of O are zero.  pre_pad: the real rows are the last
    lens[beta] rows, the sequence is pre-padded to m*b, and rows
    < N - lens[beta] of O are zero."""
    q, k, v = _f64(q, k, v)
    out = np.zeros_like(v)
    N = q.shape[2]
    for bi in range(q.shape[0]):
        n = int(lens[bi])
        assert 0 <= n <= N <= m * b
        rows = slice(N - n, N) if pre_pad else slice(0, n)
        for h in range(q.shape[1]):
            L, R = factors(q[bi, h, rows], k[bi, h, rows], m, b, T, n=n, batch_padding=True, pre_pad=pre_pad)
            out[bi, h, rows] = monarch_apply(L, R, v[bi, h, rows], pre_pad=pre_pad)
    return out


def dense_monarch(L: np.ndarray, R: np.ndarray) -> np.ndarray:
    """M from the block/entrywise form (eq. monarch_entrywise): M[l*b+j, k*b+i] = L[j,k,l] R[k,j,i]."""
    b, m, _ = L.shape
    n = m * b
    M = np.empty((n, n))
    for l in range(m):
        for j in range(b):
            for k in range(m):
                M[l * b + j, k * b: (k + 1) * b] = L[j, k, l] * R[k, j, :]
    return M


def dense_monarch_factored(L: np.ndarray, R: np.ndarray) -> np.ndarray:
    """M = P^T B with B = blockdiag(L_j^T) P blockdiag(R_k) (Sec. 2, Monarch matrices)."""
    b, m, _ = L.shape
    n = m * b
    left = np.zeros((n, n))
    for j in range(b):
        left[j * m:(j + 1) * m, j * m:(j + 1) * m] = L[j].T      # (L_j)[k, l] = L[j,k,l]
    right = np.zeros((n, n))
    for k in range(m):
        right[k * b:(k + 1) * b, k * b:(k + 1) * b] = R[k]        # (R_k)[j, i] = R[k,j,i]
    P = perm_matrix(m, b)
    return P.T @ (left @ P @ right)


def objective_dense(A: np.ndarray, q: np.ndarray, k: np.ndarray) -> float:
    """f(A; Q, K) = <A, s Q K^T> + H(A) (eq. softmax_variational_attention), 0 log 0 = 0."""
    q, k = _f64(q, k)
    s = 1.0 / np.sqrt(q.shape[1])
    return float(np.sum(A * (s * q @ k.T))) - _xlogx_sum(A)


def objective_monarch(L: np.ndarray, R: np.ndarray, q: np.ndarray, k: np.ndarray) -> float:
    """f(M; Q, K) from the factors via the separable entropy (Sec. 3, Softmax Objective):
    sum_{j,k} <Qtilde_j^T L_jk, K_k^T R_kj> + (1^T R_kj) H(L_jk) + (1^T L_jk) H(R_kj)."""
    q, k = _f64(q, k)
    b, m, _ = L.shape
    s = 1.0 / np.sqrt(q.shape[1])
    Qb = qbar(s * q, m, b)
    Kb = kbar(k, m, b)
    f = 0.0
    for j in range(b):
        for kk in range(m):
            lv, rv = L[j, kk], R[kk, j]
            f += float((Qb[j].T @ lv) @ (Kb[kk].T @ rv))
            f += rv.sum() * (-_xlogx_sum(lv)) + lv.sum() * (-_xlogx_sum(rv))
    return f


def objective_after_l_update(R: np.ndarray, q, k, m: int, b: int, n=None) -> float:
    """f(M) right after the L update that follows R, as the sum over query rows
    (j, l) of logsumexp_k of the L-update logits z[j,l,k] = <Qbar[j,l], alpha_L[j,k]>
    - c_L[j,k] (eq. L_update): the L update maximises f over L with R fixed, and
    row by row the maximum of <p, z> + H(p) over the simplex is logsumexp(z)
    (eq. softmax_variational).  q, k: one head, zero-padded to m*b rows when n < m*b;
    the sum runs over all m*b rows of the (padded) problem."""
    q, k = _f64(q, k)
    if q.shape[0] < m * b:
        q, k = pad_rows(q, m, b), pad_rows(k, m, b)
    s = 1.0 / np.sqrt(q.shape[1])
    Qb, Kb = qbar(s * q, m, b), kbar(k, m, b)
    f = 0.0
    for j in range(b):
        alpha_l = np.stack([R[kk, j] @ Kb[kk] for kk in range(m)])
        c_l = np.array([_xlogx_sum(R[kk, j]) for kk in range(m)])
        for l in range(m):
            f += log_sum_exp(alpha_l @ Qb[j, l] - c_l)
    return f


def dense_softmax_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """O = softmax(Q K^T / sqrt(d)) V, rows softmaxed (eq. softmax_attention). One head."""
    q, k, v = _f64(q, k, v)
    z = (q @ k.T) / np.sqrt(q.shape[1])
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return (e / e.sum(axis=1, keepdims=True)) @ v


def log_sum_exp(z: np.ndarray) -> float:
    (z,) = _f64(z)
    zm = z.max()
    return float(zm + np.log(np.sum(np.exp(z - zm))))
