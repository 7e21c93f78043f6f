"""The gradient pins are sharp: plant one plausible mistake at a time in the
gradient references of oracle/backward.py (on the CPU) and check that at
least one pin of test_oracle_backward.py then fails.

Mutants of the hand-derived reverse sweep replace its softmax pull-back;
mutants of the torch forward (the function autograd differentiates) are
small edits of a copy of it: a dropped entropy term, a dropped key mask, a
dropped 1/c_R, the scale applied to the keys twice.
"""
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


def _battery():
    """Names of the gradient pins that fail with the current oracle functions."""
    failed = []
    for n, m, b, T in ((12, 3, 4, 2), (10, 3, 4, 2)):   # the second one padded
        q, k, v, _ = _head(n, 6, seed=n + T)
        o = bw.torch_forward(*(torch.tensor(x) for x in (q, k, v)), m, b, T).numpy()
        if np.abs(o - nv.monarch_attention_head(q, k, v, m, b, T)).max() > 1e-12:
            failed.append(f"forward-n{n}")
    q, k, v, do = _head(8, 4, seed=28)
    for g, w in zip(bw.autograd_grads(q, k, v, do, 1, 8, 2), bw.attention_grads(q, k, v, do)):
        if np.abs(g - w).max() > 1e-12:
            failed.append("one-block")
            break
    for n, m, b, d, T in ((12, 3, 4, 5, 2), (10, 3, 4, 6, 2)):
        q, k, v, do = _head(n, d, seed=30 + n + T)
        got = bw.state_form_backward(q, k, v, do, m, b, T)
        want = bw.autograd_grads(q, k, v, do, m, b, T)
        if any(np.abs(g - w).max() > 1e-10 * max(1.0, np.abs(w).max()) for g, w in zip(got, want)):
            failed.append(f"state-form-n{n}")
    return failed


def test_unmutated_gradient_oracle_passes_battery():
    assert _battery() == []


def _softmax_back_variant(kind):
    def softmax_back(p, dp):
        if kind == "no-centering":
            return p * dp
        if kind == "plus-centering":
            return p * (dp + np.dot(dp, p))
        return dp - np.dot(dp, p)          # "no-p": the factor p dropped
    return softmax_back


def _torch_forward_variant(kind):
    """A copy of the torch forward with one mistake."""
    def torch_forward(q, k, v, m, b, T, batch_padding=False):
        assert not batch_padding  # the battery runs single sequences
        n, d = q.shape
        pad = m * b - n
        if pad:
            z = q.new_zeros(pad, d)
            q, k, v = torch.cat([q, z]), torch.cat([k, z]), torch.cat([v, z])
        s = 1.0 / np.sqrt(d)
        Qb = (s * q).reshape(m, b, d).permute(1, 0, 2)
        Kb = (s * k if kind == "scale-twice" else k).reshape(m, b, d)
        Vb = v.reshape(m, b, d)
        keymask = torch.zeros(m, 1, b, dtype=q.dtype)
        if pad and kind != "no-mask":
            pos = torch.arange(m * b).reshape(m, 1, b)
            keymask = keymask.masked_fill(pos >= n, float("-inf"))
        L = torch.eye(m, dtype=q.dtype).expand(b, m, m)
        for _ in range(T):
            alpha_r = torch.einsum("jkl,jld->kjd", L, Qb)
            c_r = L.sum(dim=2).transpose(0, 1)
            beta_r = torch.einsum("kjd,kid->kji", alpha_r, Kb)
            R = torch.softmax((beta_r if kind == "no-divide" else beta_r / c_r[..., None]) + keymask, dim=2)
            alpha_l = torch.einsum("kji,kid->jkd", R, Kb)
            live = R > 0
            c_l = torch.where(live, R * torch.log(torch.where(live, R, torch.ones_like(R))), torch.zeros_like(R))
            c_l = c_l.sum(dim=2).transpose(0, 1)
            if kind == "no-entropy":
                c_l = 0 * c_l
            beta_l = torch.einsum("jld,jkd->jlk", Qb, alpha_l)
            L = torch.softmax(beta_l - c_l[:, None, :], dim=2).permute(0, 2, 1)
        Y = torch.einsum("kji,kid->jkd", R, Vb)
        Oj = torch.einsum("jkl,jkd->jld", L, Y)
        return Oj.permute(1, 0, 2).reshape(m * b, d)[:n]
    return torch_forward


MUTANTS = {
    "sweep: softmax pull-back without centering": ("_softmax_back", lambda: _softmax_back_variant("no-centering")),
    "sweep: centering with the wrong sign": ("_softmax_back", lambda: _softmax_back_variant("plus-centering")),
    "sweep: factor p dropped": ("_softmax_back", lambda: _softmax_back_variant("no-p")),
    "forward: entropy term c_L dropped": ("torch_forward", lambda: _torch_forward_variant("no-entropy")),
    "forward: key mask dropped": ("torch_forward", lambda: _torch_forward_variant("no-mask")),
    "forward: 1/c_R dropped": ("torch_forward", lambda: _torch_forward_variant("no-divide")),
    "forward: keys scaled too": ("torch_forward", lambda: _torch_forward_variant("scale-twice")),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_gradient_mutant_is_caught(monkeypatch, name):
    attr, make = MUTANTS[name]
    monkeypatch.setattr(bw, attr, make())
    failed = _battery()
    print(name, "->", failed)
    assert failed, f"mutant '{name}' passed every gradient pin"
