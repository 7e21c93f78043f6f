"""fp64 CPU references for the gradient of the MonarchAttention forward pass.

TEST INFRASTRUCTURE ONLY: used by the test suite; the product path never
imports it.

The paper gives no gradient for the unrolled T-step iteration, so two
independent references are kept here:

* ``torch_forward`` / ``autograd_grads``: the materialised-factor algorithm
  (Sec. 3: L^(0) = I, then per step eqs. beta_r, R_update, beta_l, L_update;
  eq. monarch_multiply) written with plain PyTorch CPU ops in float64, and
  differentiated by torch.autograd.  Pinned by finite differences and, for
  m = 1, by the textbook softmax-attention gradient.
* ``state_form_backward``: reverse mode through the state form (alpha_R, c_R,
  alpha_L, c_L, Y), derived by hand below, one unit (key block k or residue
  class j) at a time -- the organisation a GPU implementation follows.

Derivation (per head, Qbar = s * Q in the layout of eq. beta_r):
  forward step t:  Z_R[k,j,i] = <alpha_R[k,j], Kbar[k,i]> / c_R[k,j] (+ omega),
                   R = softmax_i Z_R,  alpha_L[j,k] = sum_i R Kbar[k,i],
                   c_L[j,k] = sum_i R log R,
                   Z_L[j,l,k] = <Qbar[j,l], alpha_L[j,k]> - c_L[j,k],
                   L[j,k,l] = softmax_k Z_L,
                   alpha_R'[k,j] = sum_l L Qbar[j,l],  c_R'[k,j] = sum_l L;
  output:          Y[j,k] = sum_i R Vbar[k,i],  O[l*b+j] = sum_k L Y[j,k].
  A softmax p = softmax(z) pulls back dp to dz = p * (dp - <dp, p>).
  Reverse sweep: from dO, the last L update gives dL = dO . Y and dY; from
  dL the L softmax gives dZ_L, hence dQbar += dZ_L alpha_L, d alpha_L =
  dZ_L^T Qbar, d c_L = -sum_l dZ_L.  The R update of the same step gets dR =
  d alpha_L . Kbar + d c_L (log R + 1) (+ dY . Vbar at the last step),
  dKbar += R^T d alpha_L (+ dVbar = R^T dY), and through its softmax dZ_R,
  hence d alpha_R = dZ_R Kbar / c_R, dKbar += dZ_R^T alpha_R / c_R and
  d c_R = -sum_i dZ_R Z_R / c_R.  At t = 1, alpha_R[k,j] = Qbar[j,k] (the
  identity L^(0)) gives dQbar directly; for t > 1 the L update of step t-1
  gets dL = d alpha_R . Qbar + d c_R and dQbar += L d alpha_R, and the sweep
  continues.  Finally dQ = s * dQbar (rows l*b + j).

Batch padding (``batch_padding=True``): a sequence of n rows at the batch's m
and b may have whole key blocks of padding.  As in the forward oracle, such
a block has R = 0 and no L weight (Z_L = -inf), so it passes no gradient;
rows past n are inputs that the forward replaces by zero, so their
gradients are zero.
"""
from __future__ import annotations

import numpy as np
import torch


# -- the forward pass in torch (for autograd) ---------------------------------------------

def torch_forward(q, k, v, m: int, b: int, T: int, batch_padding: bool = False):
    """O for one head; q, k, v float64 torch tensors [N, d], N <= m*b (post-padding;
    with batch_padding any 1 <= N <= m*b, whole blocks of padding allowed)."""
    n, d = q.shape
    if batch_padding:
        assert 1 <= n <= m * b and T >= 1
    else:
        assert (m - 1) * b < n <= m * b and T >= 1
    pad = m * b - n
    if pad:
        z = q.new_zeros(pad, d)
        q, k, v = torch.cat([q, z]), torch.cat([k, z]), torch.cat([v, z])
    s = 1.0 / np.sqrt(d)
    Qb = (s * q).reshape(m, b, d).permute(1, 0, 2)       # Qbar[j, l] = s * Q[l*b + j]
    Kb = k.reshape(m, b, d)                              # Kbar[k, i] = K[k*b + i]
    Vb = v.reshape(m, b, d)
    keymask = torch.zeros(m, 1, b, dtype=q.dtype)        # omega over i, by block k
    if pad:
        pos = torch.arange(m * b).reshape(m, 1, b)
        keymask = keymask.masked_fill(pos >= n, float("-inf"))
    live = -(-n // b)                                    # key blocks with a real key
    empty = (torch.arange(m) >= live)[:, None, None]     # blocks of padding only: R = 0
    keymask = keymask.masked_fill(empty, 0.0)            # (their softmax input is kept finite)
    lmask = torch.zeros(m, dtype=q.dtype).masked_fill(torch.arange(m) >= live, float("-inf"))
    L = torch.eye(m, dtype=q.dtype).expand(b, m, m)      # L^(0)[j, k, l] = delta_kl
    for _ in range(T):
        alpha_r = torch.einsum("jkl,jld->kjd", L, Qb)    # eq. beta_r
        c_r = L.sum(dim=2).transpose(0, 1)               # [k, j]
        c_r = torch.where(empty[:, :, 0], torch.ones_like(c_r), c_r)   # zero (unused) on empty blocks
        beta_r = torch.einsum("kjd,kid->kji", alpha_r, Kb)
        R = torch.softmax(beta_r / c_r[..., None] + keymask, dim=2)      # eq. R_update
        R = torch.where(empty, torch.zeros_like(R), R)
        alpha_l = torch.einsum("kji,kid->jkd", R, Kb)    # eq. beta_l
        # sum_i R log R over the real keys (masked entries are exactly 0 and
        # contribute 0; the inner where keeps log away from them, also in the gradient)
        live = R > 0
        c_l = torch.where(live, R * torch.log(torch.where(live, R, torch.ones_like(R))), torch.zeros_like(R))
        c_l = c_l.sum(dim=2).transpose(0, 1)                               # [j, k]
        beta_l = torch.einsum("jld,jkd->jlk", Qb, alpha_l)
        L = torch.softmax(beta_l - c_l[:, None, :] + lmask, dim=2).permute(0, 2, 1)  # eq. L_update, [j, k, l]
    Y = torch.einsum("kji,kid->jkd", R, Vb)              # eq. monarch_multiply
    Oj = torch.einsum("jkl,jkd->jld", L, Y)              # O[l*b + j] = Oj[j, l]
    return Oj.permute(1, 0, 2).reshape(m * b, d)[:n]


def autograd_grads(q, k, v, dout, m: int, b: int, T: int, batch_padding: bool = False):
    """(dQ, dK, dV) of <O, dout> for one head, numpy float64 arrays in and out
    (with batch_padding, n = 0 rows gives empty gradients)."""
    if q.shape[0] == 0:
        return (np.zeros((0, q.shape[1])),) * 3
    tq, tk, tv = (torch.tensor(np.asarray(x, dtype=np.float64), requires_grad=True) for x in (q, k, v))
    o = torch_forward(tq, tk, tv, m, b, T, batch_padding)
    gq, gk, gv = torch.autograd.grad(o, (tq, tk, tv), torch.tensor(np.asarray(dout, dtype=np.float64)))
    return gq.numpy(), gk.numpy(), gv.numpy()


def attention_grads(q, k, v, dout):
    """The textbook gradient of exact softmax attention O = softmax(s Q K^T) V."""
    q, k, v, dout = (np.asarray(x, dtype=np.float64) for x in (q, k, v, dout))
    s = 1.0 / np.sqrt(q.shape[1])
    z = s * q @ k.T
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    dv = p.T @ dout
    dp = dout @ v.T
    dz = p * (dp - (dp * p).sum(axis=1, keepdims=True))
    return s * dz @ k, s * dz.T @ q, dv


# -- reverse mode through the state form ---------------------------------------------------

def _softmax(z):
    e = np.exp(z - z.max())
    return e / e.sum()


def _softmax_back(p, dp):
    return p * (dp - np.dot(dp, p))


def state_form_backward(q, k, v, dout, m: int, b: int, T: int, batch_padding: bool = False):
    """(dQ, dK, dV) for one head by the reverse sweep of the module docstring."""
    q, k, v, dout = (np.asarray(x, dtype=np.float64) for x in (q, k, v, dout))
    n, d = q.shape
    if batch_padding:
        assert 0 <= n <= m * b
    else:
        assert (m - 1) * b < n <= m * b
    Np = m * b
    qp, kp, vp, dop = (np.zeros((Np, d)) for _ in range(4))
    qp[:n], kp[:n], vp[:n], dop[:n] = q, k, v, dout
    s = 1.0 / np.sqrt(d)
    Qb = np.stack([np.stack([s * qp[l * b + j] for l in range(m)]) for j in range(b)])  # [j, l, d]
    Kb = kp.reshape(m, b, d)
    Vb = vp.reshape(m, b, d)
    nkeys = [max(min(b, n - kk * b), 0) for kk in range(m)]   # 0: a block of padding only
    live = -(-n // b)                                          # blocks with a real key

    # forward, keeping the states of every step
    aR = [np.stack([np.stack([Qb[j, kk] for j in range(b)]) for kk in range(m)])]   # alpha_R^(1)[k, j]
    cR = [np.ones((m, b))]
    aL, cL, Rs, Ls = [], [], [], []
    for t in range(T):
        R = np.zeros((m, b, b))
        for kk in range(live):
            for j in range(b):
                z = Kb[kk, : nkeys[kk]] @ aR[t][kk, j] / cR[t][kk, j]
                R[kk, j, : nkeys[kk]] = _softmax(z)
        al = np.einsum("kji,kid->jkd", R, Kb)
        cl = np.zeros((b, m))
        for kk in range(m):
            for j in range(b):
                r = R[kk, j][R[kk, j] > 0]
                cl[j, kk] = np.sum(r * np.log(r))
        L = np.zeros((b, m, m))
        for j in range(b):
            for l in range(m):
                if live:
                    L[j, :live, l] = _softmax((al[j] @ Qb[j, l] - cl[j])[:live])
        Rs.append(R), aL.append(al), cL.append(cl), Ls.append(L)
        if t + 1 < T:
            aR.append(np.einsum("jkl,jld->kjd", L, Qb))
            cR.append(L.sum(axis=2).T.copy())
    Y = np.einsum("kji,kid->jkd", Rs[-1], Vb)

    dQb = np.zeros_like(Qb)
    dKb = np.zeros_like(Kb)
    dVb = np.zeros_like(Vb)
    dOj = np.stack([np.stack([dop[l * b + j] for l in range(m)]) for j in range(b)])   # [j, l, d]

    # the last L update and the output
    L = Ls[-1]
    dY = np.einsum("jkl,jld->jkd", L, dOj)
    dL = np.einsum("jld,jkd->jkl", dOj, Y)
    daR = dcR = None
    for t in range(T - 1, -1, -1):
        L, al, cl, R = Ls[t], aL[t], cL[t], Rs[t]
        if t < T - 1:   # the L update of step t feeds alpha_R, c_R of step t+1
            dL = np.einsum("kjd,jld->jkl", daR, Qb) + dcR.T[:, :, None]
            dQb += np.einsum("jkl,kjd->jld", L, daR)
        # L softmax over k, per (j, l)
        dal = np.zeros_like(al)
        dcl = np.zeros_like(cl)
        for j in range(b):
            for l in range(m):
                dz = _softmax_back(L[j, :, l], dL[j, :, l])   # zero on the blocks left out
                dQb[j, l] += dz @ al[j]
                dal[j] += np.outer(dz, Qb[j, l])
                dcl[j] -= dz
        # R update of step t
        daR = np.zeros((m, b, d))
        dcR = np.zeros((m, b))
        for kk in range(live):      # blocks of padding only have R = 0 and pass nothing back
            nk = nkeys[kk]
            for j in range(b):
                r = R[kk, j, :nk]
                drr = Kb[kk, :nk] @ dal[j, kk] + dcl[j, kk] * (np.log(r) + 1.0)
                if t == T - 1:
                    drr = drr + Vb[kk, :nk] @ dY[j, kk]
                    dVb[kk, :nk] += np.outer(r, dY[j, kk])
                dKb[kk, :nk] += np.outer(r, dal[j, kk])
                dz = _softmax_back(r, drr)
                c = cR[t][kk, j]
                zr = Kb[kk, :nk] @ aR[t][kk, j] / c
                daR[kk, j] = dz @ Kb[kk, :nk] / c
                dKb[kk, :nk] += np.outer(dz, aR[t][kk, j]) / c
                dcR[kk, j] = -np.dot(dz, zr) / c
        if t == 0:   # alpha_R^(1)[k, j] = Qbar[j, k]; c_R^(1) = 1 is a constant
            for kk in range(m):
                for j in range(b):
                    dQb[j, kk] += daR[kk, j]
    dq = np.zeros((Np, d))
    for j in range(b):
        for l in range(m):
            dq[l * b + j] = s * dQb[j, l]
    return dq[:n], dKb.reshape(Np, d)[:n], dVb.reshape(Np, d)[:n]
