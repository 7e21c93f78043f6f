"""Calls captured into HIP graphs (torch.cuda.graph).

A captured call bakes its workspace address into the graph.  The library
therefore refuses to allocate under capture (the stream's workspace must be
sized by an earlier call on it), and never frees a buffer that a capture
used until monarch_attn_release_workspace.  Every replay is checked against
an eager call on the same inputs (the same kernels and grids, so bitwise),
with the program's own eager work and synchronisations between replays.
"""
import numpy as np
import pytest

import oracle
import synth_inputs as si

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ma():
    import torch

    assert torch.cuda.is_available(), "no GPU visible"
    import paper_2505_18698_amd as ma

    return ma


def _inputs(B, H, N, d, seed, n_sets):
    import torch

    sets = []
    for r in range(n_sets):
        q, k, v = si.random_qkv(B, H, N, d, "bf16", seed=seed + r, scale=1.5)
        sets.append([torch.from_numpy(x).to(torch.bfloat16).cuda() for x in (q, k, v)])
    return sets


def _warm_and_capture(fn, stream):
    """One eager call on `stream` (it sizes the stream's workspace), then a
    graph of the same call captured on it."""
    import torch

    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        fn()
    stream.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("path,N,m,b,T", [("half_steps", 1024, 32, 32, 2), ("half_steps", 300, 19, 16, 3),
                                          ("auto", 196, 14, 14, 2)])
def test_captured_forward_replays_match_eager(ma, path, N, m, b, T):
    import torch

    prev = ma.monarch_attn_set_path(ma.PATH_HALF_STEPS if path == "half_steps" else ma.PATH_AUTO)
    try:
        B, H, d = 2, 4, 64
        sets = _inputs(B, H, N, d, seed=500 + N, n_sets=3)
        q, k, v = (t.clone() for t in sets[0])
        out = torch.full_like(q, float("nan"))
        g = _warm_and_capture(lambda: ma.monarch_attn_fwd(q, k, v, out, m, b, T), torch.cuda.Stream())
        for r, (qs, ks, vs) in enumerate(sets + sets[:1]):
            q.copy_(qs), k.copy_(ks), v.copy_(vs)
            out.fill_(float("nan"))
            g.replay()
            torch.cuda.synchronize()
            eager = torch.full_like(q, float("nan"))
            ma.monarch_attn_fwd(q, k, v, eager, m, b, T)
            torch.cuda.synchronize()
            print(f"{path} N={N} replay {r}: bitwise equal to eager", flush=True)
            assert torch.equal(out, eager), (path, N, r)
            ref = oracle.monarch_attention(*(x.float().cpu().numpy() for x in (qs, ks, vs)), m, b, T)
            assert oracle.rel_frobenius(out.double().cpu().numpy(), ref) <= 2e-2
        del g
    finally:
        ma.monarch_attn_set_path(prev)


def test_captured_gradient_replays_match_eager(ma):
    import torch

    B, H, N, d, m, b, T = 1, 4, 1024, 64, 32, 32, 2
    sets = _inputs(B, H, N, d, seed=600, n_sets=2)
    q, k, v = (t.clone() for t in sets[0])
    do = torch.from_numpy(si.random_cotangent((B, H, N, d), "bf16", seed=601)).to(torch.bfloat16).cuda()
    grads = [torch.empty_like(q) for _ in range(3)]
    g = _warm_and_capture(lambda: ma.monarch_attn_bwd(q, k, v, do, *grads, m, b, T), torch.cuda.Stream())
    for r, (qs, ks, vs) in enumerate(sets + sets[:1]):
        q.copy_(qs), k.copy_(ks), v.copy_(vs)
        for x in grads:
            x.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        eager = [torch.empty_like(q) for _ in range(3)]
        ma.monarch_attn_bwd(q, k, v, do, *eager, m, b, T)
        torch.cuda.synchronize()
        print(f"gradient replay {r}: bitwise equal to eager", flush=True)
        for x, y in zip(grads, eager):
            assert torch.equal(x, y), r
    del g


def test_capture_with_a_small_workspace_fails_cleanly(ma):
    """On a stream whose workspace was never sized, a captured call neither
    allocates nor launches: it fails with MA_EUNSUPPORTED, and the same call
    runs eagerly afterwards."""
    import torch

    prev = ma.monarch_attn_set_path(ma.PATH_HALF_STEPS)
    try:
        B, H, N, d, m, b, T = 1, 2, 256, 64, 16, 16, 2
        (q, k, v), = _inputs(B, H, N, d, seed=700, n_sets=1)
        out = torch.full_like(q, float("nan"))
        # torch hands out streams from a pool: free every stream's workspace
        # (no graph of this process is alive) so that this one is empty
        torch.cuda.synchronize()
        ma.monarch_attn_release_workspace()
        s = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        ticks = torch.zeros(1, device="cuda")
        with pytest.raises(ma.MonarchAttnError) as err:
            with torch.cuda.graph(g, stream=s):
                ticks.add_(1)  # the graph is not empty
                ma.monarch_attn_fwd(q, k, v, out, m, b, T)
        assert err.value.status == ma.MA_EUNSUPPORTED and "being captured" in str(err.value), err.value
        torch.cuda.synchronize()
        assert torch.isnan(out).all()
        with torch.cuda.stream(s):
            ma.monarch_attn_fwd(q, k, v, out, m, b, T)
        torch.cuda.synchronize()
        ref = oracle.monarch_attention(*(x.float().cpu().numpy() for x in (q, k, v)), m, b, T)
        assert oracle.rel_frobenius(out.double().cpu().numpy(), ref) <= 2e-2
    finally:
        ma.monarch_attn_set_path(prev)


def test_workspace_growth_keeps_a_captured_buffer(ma):
    """A larger eager call on the capture stream grows its workspace; the
    buffer the graph holds stays allocated, so later replays still match."""
    import torch

    prev = ma.monarch_attn_set_path(ma.PATH_HALF_STEPS)
    try:
        m, b, T, d = 16, 16, 2, 64
        (q, k, v), = _inputs(1, 2, 256, d, seed=800, n_sets=1)
        out = torch.full_like(q, float("nan"))
        s = torch.cuda.Stream()
        g = _warm_and_capture(lambda: ma.monarch_attn_fwd(q, k, v, out, m, b, T), s)
        (q2, k2, v2), = _inputs(4, 8, 4096, d, seed=801, n_sets=1)
        out2 = torch.empty_like(q2)
        with torch.cuda.stream(s):  # needs a workspace 64x as large
            ma.monarch_attn_fwd(q2, k2, v2, out2, 64, 64, T)
        torch.cuda.synchronize()
        scratch = torch.randn(64 << 20, device="cuda")  # new allocations may land anywhere freed
        for r in range(3):
            out.fill_(float("nan"))
            g.replay()
            torch.cuda.synchronize()
            eager = torch.empty_like(q)
            ma.monarch_attn_fwd(q, k, v, eager, m, b, T)
            torch.cuda.synchronize()
            assert torch.equal(out, eager), r
        del g, scratch
    finally:
        ma.monarch_attn_set_path(prev)


def test_timing_cannot_be_captured(ma):
    import torch

    B, H, N, d, m, b, T = 1, 2, 256, 64, 16, 16, 2
    (q, k, v), = _inputs(B, H, N, d, seed=900, n_sets=1)
    out = torch.empty_like(q)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        ma.monarch_attn_fwd(q, k, v, out, m, b, T)
    s.synchronize()
    ma.monarch_attn_timing_enable(True)
    try:
        g = torch.cuda.CUDAGraph()
        ticks = torch.zeros(1, device="cuda")
        with pytest.raises(ma.MonarchAttnError) as err:
            with torch.cuda.graph(g, stream=s):
                ticks.add_(1)
                ma.monarch_attn_fwd(q, k, v, out, m, b, T)
        assert err.value.status == ma.MA_EUNSUPPORTED and "timing" in str(err.value)
    finally:
        ma.monarch_attn_timing_enable(False)
    torch.cuda.synchronize()
    assert np.isfinite(out.float().cpu().numpy()).all()


@pytest.mark.parametrize("entry", ["varlen", "objective", "exact"])
def test_other_entry_points_replay_match_eager(ma, entry):
    """The padded-batch, objective and exact-attention calls under capture."""
    import torch

    B, H, N, d, m, b, T = 3, 2, 640, 64, 20, 32, 2
    sets = _inputs(B, H, N, d, seed=1000, n_sets=2)
    q, k, v = (t.clone() for t in sets[0])
    lens = torch.tensor([640, 333, 17], dtype=torch.int32, device="cuda")
    out = torch.empty_like(q)
    aux = torch.empty(B, H, T if entry == "objective" else N, dtype=torch.float32, device="cuda")

    def call(o, a):
        if entry == "varlen":
            ma.monarch_attn_fwd_varlen(q, k, v, o, lens, m, b, T)
        elif entry == "objective":
            ma.monarch_attn_fwd_objective(q, k, v, o, a, m, b, T)
        else:
            ma.monarch_attn_exact_fwd(q, k, v, o, a)

    g = _warm_and_capture(lambda: call(out, aux), torch.cuda.Stream())
    for r, (qs, ks, vs) in enumerate(sets + sets[:1]):
        q.copy_(qs), k.copy_(ks), v.copy_(vs)
        out.fill_(float("nan")), aux.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        eo, ea = torch.full_like(out, float("nan")), torch.full_like(aux, float("nan"))
        call(eo, ea)
        torch.cuda.synchronize()
        print(f"{entry} replay {r}: bitwise equal to eager", flush=True)
        assert torch.equal(out, eo), (entry, r)
        if entry != "varlen":  # the padded-batch call has no second output
            assert torch.equal(aux, ea), (entry, r)
    del g
