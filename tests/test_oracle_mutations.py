"""The pins are sharp: plant one plausible mistake in the (numpy) oracle at a
time, on the CPU, and check that at least one pin then fails.

Each mutant is a small edit of one update of the materialised-factor oracle
(a dropped term, a wrong sign, a transposed index, a wrong initialisation).
The pin battery below re-runs the paper-derived checks of
test_oracle_pins.py against the mutated functions.
"""
import numpy as np
import pytest

import oracle.naive as nv
import synth_inputs as si


def _head(m, b, d, seed, scale=2.0):
    q, k, v = si.random_qkv(1, 1, m * b, d, "f32", seed=seed, scale=scale)
    return q[0, 0].astype(np.float64), k[0, 0].astype(np.float64), v[0, 0].astype(np.float64)


def _battery():
    """Return the names of the pins that fail with the current oracle functions."""
    failed = []
    # permutation worked example
    x = np.arange(1.0, 7.0)
    if not np.array_equal(nv.qbar(x[:, None], 2, 3).reshape(-1), np.array([1, 4, 2, 5, 3, 6.0])):
        failed.append("perm")
    # block maximisers and ascent, T = 2 and 3
    for T in (2, 3):
        m, b = 3, 4
        q, k, v = _head(m, b, 5, seed=100 + T)
        try:
            L, R, hist = nv.factors(q, k, m, b, T, history=True)
        except Exception:
            failed.append("crash")
            continue
        M = nv.dense_monarch(L, R)
        if not (np.all(M >= -1e-15) and np.allclose(M.sum(axis=1), 1.0, atol=1e-12)):
            failed.append("stochastic")
        vals = [nv.objective_dense(nv.dense_monarch(Lh, Rh), q, k) for Lh, Rh in hist[1:]]
        if any(b2 < a2 - 1e-12 for a2, b2 in zip(vals, vals[1:])):
            failed.append("ascent")
        rng = np.random.default_rng(T)
        Lp, Rl = hist[-2]
        f_r = nv.objective_dense(nv.dense_monarch(Lp, Rl), q, k)
        f_l = nv.objective_dense(nv.dense_monarch(L, R), q, k)
        for _ in range(30):
            kk, j = rng.integers(m), rng.integers(b)
            R2 = Rl.copy()
            R2[kk, j] = 0.99 * R2[kk, j] + 0.01 * rng.dirichlet(np.ones(b))
            if nv.objective_dense(nv.dense_monarch(Lp, R2), q, k) > f_r + 1e-12:
                failed.append("R-maximiser")
                break
        for _ in range(30):
            j, l = rng.integers(b), rng.integers(m)
            L2 = L.copy()
            L2[j, :, l] = 0.99 * L2[j, :, l] + 0.01 * rng.dirichlet(np.ones(m))
            if nv.objective_dense(nv.dense_monarch(L2, R), q, k) > f_l + 1e-12:
                failed.append("L-maximiser")
                break
    # special cases
    for (m, b, T) in ((1, 6, 2), (6, 1, 2)):
        q, k, v = _head(m, b, 4, seed=200)
        o = nv.monarch_attention_head(q, k, v, m, b, T)
        if np.abs(o - nv.dense_softmax_attention(q, k, v)).max() > 1e-12:
            failed.append(f"exact-m{m}-b{b}")
    q, k, v = _head(4, 3, 4, seed=300)
    q[:] = q[0]
    if np.abs(nv.monarch_attention_head(q, k, v, 4, 3, 2) - nv.dense_softmax_attention(q, k, v)).max() > 1e-12:
        failed.append("identical-queries")
    q, k, v = _head(4, 3, 4, seed=301)
    if np.abs(nv.monarch_attention_head(q, 0 * k, v, 4, 3, 2) - v.mean(axis=0)).max() > 1e-12:
        failed.append("zero-keys")
    # key-block permutation is not a symmetry (L^(0) = I pairs query block l with key block l)
    q, k, v = _head(4, 3, 4, seed=302)
    perm = np.concatenate([np.arange(3, 6), np.arange(0, 3), np.arange(6, 12)])
    o1 = nv.monarch_attention_head(q, k, v, 4, 3, 1)
    o2 = nv.monarch_attention_head(q, k[perm], v[perm], 4, 3, 1)
    if np.abs(o1 - o2).max() < 1e-6:
        failed.append("block-symmetry")
    # apply against the dense matrix
    m, b = 3, 4
    q, k, v = _head(m, b, 5, seed=400)
    L, R = nv.factors(q, k, m, b, 2)
    if np.abs(nv.monarch_apply(L, R, v) - nv.dense_monarch(L, R) @ v).max() > 1e-12:
        failed.append("apply")
    failed += _padding_battery()
    failed += _batch_padding_battery()
    return failed


def _batch_padding_battery():
    """Pins of the batch-padding reading (whole key blocks of padding)."""
    import oracle
    failed = []
    try:
        # b = 1: exact attention over the real keys, T = 2
        N = 8
        q, k, v = _head(N, 1, 4, seed=600)
        o = nv.monarch_attention_varlen(q[None, None], k[None, None], v[None, None], [5], N, 1, 2)[0, 0]
        if np.abs(o[:5] - nv.dense_softmax_attention(q[:5], k[:5], v[:5])).max() > 1e-12 or np.any(o[5:] != 0):
            failed.append("varlen-exact-b1")
        # T = 1: the same real rows as the problem without the empty blocks
        m, b, n = 4, 3, 5
        q, k, v = _head(m, b, 5, seed=601)
        o = nv.monarch_attention_varlen(q[None, None], k[None, None], v[None, None], [n], m, b, 1)[0, 0]
        if np.abs(o[:n] - nv.monarch_attention_head(q[:n], k[:n], v[:n], 2, b, 1)).max() > 1e-12:
            failed.append("varlen-fewer-blocks")
        # M row-stochastic with zero padded columns
        L, R = nv.factors(q[:n], k[:n], m, b, 2, n=n, batch_padding=True)
        M = nv.dense_monarch(L, R)
        if not (np.all(M >= 0) and np.all(M[:, n:] == 0) and np.allclose(M.sum(axis=1), 1.0, atol=1e-12)):
            failed.append("varlen-stochastic")
        # the state form in C agrees (T = 2)
        ref = oracle.monarch_attention_varlen(q[None, None], k[None, None], v[None, None], np.array([n]), m, b, 2)
        o2 = nv.monarch_attention_varlen(q[None, None], k[None, None], v[None, None], [n], m, b, 2)
        if np.abs(o2 - ref).max() > 1e-12:
            failed.append("varlen-two-forms")
    except Exception:
        failed.append("varlen-crash")
    return failed


def _padding_battery():
    """Pins of Appendix "Padding and Masking" (N = 10 < m*b = 12)."""
    failed = []
    m, b, n = 3, 4, 10
    q, k, v = _head(m, b, 5, seed=500)
    q, k, v = q[:n], k[:n], v[:n]
    try:
        L, R = nv.factors(q, k, m, b, 2)
    except Exception:
        return ["pad-crash"]
    M = nv.dense_monarch(L, R)
    if np.abs(M[:, n:]).max() != 0.0 or not np.allclose(M.sum(axis=1), 1.0, atol=1e-12):
        failed.append("pad-columns")
    # explicit zero padding (rows >= n given by the caller) equals the automatic one
    qz, kz = np.zeros((m * b, 5)), np.zeros((m * b, 5))
    qz[:n], kz[:n] = q, k
    L2, R2 = nv.factors(qz, kz, m, b, 2, n=n)
    if np.abs(L2 - L).max() > 1e-15 or np.abs(R2 - R).max() > 1e-15:
        failed.append("pad-value")
    # any values in the padded key rows: same factors
    kg = kz.copy()
    kg[n:] = np.random.default_rng(1).normal(size=(m * b - n, 5)) * 3
    L3, R3 = nv.factors(qz, kg, m, b, 2, n=n)
    if np.abs(L3 - L).max() > 1e-12 or np.abs(R3 - R).max() > 1e-12:
        failed.append("pad-keys")
    # one block: exact softmax attention over the n real tokens
    q1, k1, v1 = _head(1, 8, 4, seed=501)
    o1 = nv.monarch_attention_head(q1[:5], k1[:5], v1[:5], 1, 8, 2)
    if o1.shape != (5, 4) or np.abs(o1 - nv.dense_softmax_attention(q1[:5], k1[:5], v1[:5])).max() > 1e-12:
        failed.append("pad-exact")
    return failed


def test_unmutated_oracle_passes_battery():
    assert _battery() == []


def _softmax(z):
    e = np.exp(z - z.max())
    return e / e.sum()


def _r_update_variant(kind):
    def r_update(L, Qb, Kb, omega=None):
        b, m, _ = L.shape
        R = np.empty((m, b, b))
        if omega is not None and kind == "mask-front":       # the pre-padding side
            omega = omega.reshape(-1)[::-1].reshape(m, b)
        for k in range(m):
            om = 0.0 if omega is None or kind == "no-mask" else omega[k]
            for j in range(b):
                if np.all(np.isneginf(om)):
                    R[k, j] = 0.0
                    continue
                a = L[j, k, :] @ Qb[j]
                c = L[j, k, :].sum()
                beta = Kb[k] @ a
                if kind == "no-divide":
                    R[k, j] = _softmax(beta + om)
                elif kind == "times-c":
                    R[k, j] = _softmax(beta * c + om)
                elif kind == "transposed-L":
                    R[k, j] = _softmax((Kb[k] @ (L[j, :, k] @ Qb[j])) / L[j, :, k].sum() + om)
                else:
                    R[k, j] = _softmax(beta / c + om)
        return R
    return r_update


def _l_update_variant(kind):
    def l_update(R, Qb, Kb, live=None):
        m, b, _ = R.shape
        live = m if live is None or kind == "empty-blocks-weighted" else live
        L = np.zeros((b, m, m))
        if live == 0:
            return L
        for j in range(b):
            al = np.stack([R[k, j] @ Kb[k] for k in range(m)])
            cl = np.array([np.sum(R[k, j][R[k, j] > 0] * np.log(R[k, j][R[k, j] > 0])) for k in range(m)])
            if kind == "plus-c":
                cl = -cl
            elif kind == "no-c":
                cl = 0 * cl
            for l in range(m):
                z = al @ Qb[j, l] - cl
                L[j, :live, l] = _softmax(z[:live])
            if kind == "softmax-over-l":
                for k in range(live):
                    L[j, k, :] = _softmax(np.array([al[k] @ Qb[j, l] - cl[k] for l in range(m)]))
        return L
    return l_update


def _apply_transposed(L, R, v, pre_pad=False):
    return nv.__dict__["_orig_apply"](np.transpose(L, (0, 2, 1)).copy(), R, v, pre_pad=pre_pad)


def _qbar_wrong(q, m, b):
    n, d = q.shape
    return q.reshape(b, m, d).copy()      # rows j*m + l instead of l*b + j


def _factors_uniform_init(q, k, m, b, T, *, history=False, n=None, batch_padding=False, pre_pad=False):
    rows, d = q.shape
    n = rows if n is None else n
    if rows < m * b:
        q, k = nv.pad_rows(q, m, b), nv.pad_rows(k, m, b)
    omega = nv.key_mask(n, m, b) if n < m * b else None
    live = nv.live_blocks(n, b)
    s = 1.0 / np.sqrt(d)
    Qb, Kb = nv.qbar(s * q, m, b), nv.kbar(k, m, b)
    L = np.full((b, m, m), 1.0 / m)
    hist = [(L, None)]
    for _ in range(T):
        R = nv.r_update(L, Qb, Kb, omega)
        hist.append((L, R))
        L = nv.l_update(R, Qb, Kb, live)
        hist.append((L, R))
    return (L, R, hist) if history else (L, R)


MUTANTS = {
    "R: drop the 1/c_R": ("r_update", lambda: _r_update_variant("no-divide")),
    "R: multiply by c_R": ("r_update", lambda: _r_update_variant("times-c")),
    "R: transposed L index": ("r_update", lambda: _r_update_variant("transposed-L")),
    "L: add c_L": ("l_update", lambda: _l_update_variant("plus-c")),
    "L: drop c_L": ("l_update", lambda: _l_update_variant("no-c")),
    "L: softmax over l": ("l_update", lambda: _l_update_variant("softmax-over-l")),
    "apply: transposed L": ("monarch_apply", lambda: _apply_transposed),
    "layout: wrong permutation": ("qbar", lambda: _qbar_wrong),
    "init: uniform L0": ("factors", lambda: _factors_uniform_init),
    "padding: mask omitted": ("r_update", lambda: _r_update_variant("no-mask")),
    "padding: mask on the pre-padding side": ("r_update", lambda: _r_update_variant("mask-front")),
    "padding: padded with ones": ("pad_rows", lambda: _pad_ones),
    "batch padding: empty blocks keep L weight": ("l_update", lambda: _l_update_variant("empty-blocks-weighted")),
    "batch padding: partial block dropped": ("live_blocks", lambda: (lambda n, b: n // b)),
    "batch padding: padded query rows dropped": ("monarch_attention_varlen", lambda: _varlen_fewer_blocks),
}


def _varlen_fewer_blocks(q, k, v, lens, m, b, T):
    """Each sequence solved with m = ceil(n / b), leaving out the all-padding query rows."""
    out = np.zeros_like(np.asarray(v, dtype=np.float64))
    for bi, n in enumerate(lens):
        for h in range(q.shape[1]):
            if n > 0:
                out[bi, h, :n] = nv.monarch_attention_head(q[bi, h, :n], k[bi, h, :n], v[bi, h, :n], -(-n // b), b, T)
    return out


def _pad_ones(x, m, b):
    out = np.ones((m * b,) + x.shape[1:])
    out[: x.shape[0]] = x
    return out


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_each_mutant_is_caught(monkeypatch, name):
    attr, make = MUTANTS[name]
    monkeypatch.setitem(nv.__dict__, "_orig_apply", nv.monarch_apply)
    monkeypatch.setattr(nv, attr, make())
    with np.errstate(all="ignore"):
        failed = _battery()
    assert failed, f"mutant {name!r} passed every pin"
