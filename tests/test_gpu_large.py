"""Maximum sizes: tensors of more than 2^31 elements (every offset must be
64-bit).  Inputs are drawn on the device from a seeded torch generator; the
oracle checks the first head, the head that starts exactly at element 2^31
(where a 32-bit offset would wrap) and the last head.  Needs about 31 GB
(forward) and 85 GB (gradient) of device memory."""
import numpy as np
import pytest

import oracle
import oracle.backward as ob

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ma():
    import torch

    assert torch.cuda.is_available(), "no GPU visible"
    import paper_2505_18698_amd as lib

    return lib


def _draw(torch, shape, seed, scale=1.0):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    x = torch.empty(shape, device="cuda", dtype=torch.bfloat16)
    for h in range(shape[1]):  # one head at a time: no float32 copy of the whole tensor
        x[0, h] = (scale * torch.randn(shape[2:], generator=g, device="cuda")).to(torch.bfloat16)
    return x


def _need(torch, gib):
    free, _ = torch.cuda.mem_get_info()
    if free < gib * (1 << 30):
        pytest.skip(f"needs {gib} GiB of free device memory")


def test_forward_beyond_2_to_the_31_elements(ma):
    import torch

    H, N, d, m, b, T = 1040, 16384, 128, 128, 128, 2
    assert H * N * d > 2 ** 31
    _need(torch, 40)
    q, k, v = (_draw(torch, (1, H, N, d), seed=s) for s in (1, 2, 3))
    out = torch.empty_like(q)
    ma.monarch_attn_fwd(q, k, v, out, m, b, T)
    torch.cuda.synchronize()
    heads = [0, 2 ** 31 // (N * d), H - 1]
    for h in heads:
        qs, ks, vs = (x[:, h:h + 1].float().cpu().numpy() for x in (q, k, v))
        ref = oracle.monarch_attention(qs, ks, vs, m, b, T)
        got = out[:, h:h + 1].double().cpu().numpy()
        err = oracle.rel_frobenius(got, ref)
        print(f"head {h} (first element {h * N * d}): rel_frob {err:.3e}", flush=True)
        assert np.isfinite(got).all() and err <= 2e-2
    del q, k, v, out
    torch.cuda.empty_cache()


def test_gradient_beyond_2_to_the_31_elements(ma):
    import torch

    H, N, d, m, b, T = 2100, 16384, 64, 128, 128, 1
    assert H * N * d > 2 ** 31
    _need(torch, 100)
    q, k, v, g = (_draw(torch, (1, H, N, d), seed=s) for s in (4, 5, 6, 7))
    grads = [torch.empty_like(q) for _ in range(3)]
    ma.monarch_attn_bwd(q, k, v, g, *grads, m, b, T)
    torch.cuda.synchronize()
    for h in [2 ** 31 // (N * d), H - 1]:
        qs, ks, vs, gs = (x[0, h].float().cpu().numpy() for x in (q, k, v, g))
        ref = ob.autograd_grads(qs, ks, vs, gs, m, b, T)
        errs = [oracle.rel_frobenius(x[0, h].double().cpu().numpy(), r) for x, r in zip(grads, ref)]
        print(f"head {h} (first element {h * N * d}): rel_frob dq={errs[0]:.3e} dk={errs[1]:.3e} dv={errs[2]:.3e}",
              flush=True)
        assert max(errs) <= 3e-2
    del q, k, v, g, grads
    torch.cuda.empty_cache()
    ma.monarch_attn_release_workspace()
