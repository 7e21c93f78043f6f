"""GPU parity of pre-padded sequences (monarch_attn_fwd_prepad) against the
fp64 oracle's pre-padding, which places the real rows last and masks the
keys below m*b - N (Appendix "Padding and Masking").

The kernels run the post-padded problem on rows read and written in reverse
order, so besides the oracle bar (1e-5 fp32, 2e-2 bf16/fp16, and twice that
per residue class) the result equals the post-padded call on the
row-reversed tensors, row-reversed, bit for bit.  Every tensor is followed by
NaN guard rows, and the rows of a left-padded batch before its real ones
hold NaN: neither may reach the output.
"""
import numpy as np
import pytest

import oracle
import parity
import synth_inputs as si

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2, "f16": 2e-2}
GUARD = 4096


@pytest.fixture(scope="module")
def lib():
    import torch

    assert torch.cuda.is_available(), "no GPU visible"
    import paper_2505_18698_amd as ma

    return ma


@pytest.fixture(params=["half_steps", "fused"])
def ma(lib, request):
    prev = lib.monarch_attn_set_path(lib.PATH_HALF_STEPS if request.param == "half_steps" else lib.PATH_FUSED)
    lib.path_name = request.param
    yield lib
    lib.monarch_attn_set_path(prev)


def _td(dtype):
    import torch

    return {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]


def _guarded(torch, x, td):
    flat = torch.full((x.size + GUARD,), float("nan"), dtype=td, device="cuda")
    flat[: x.size].copy_(torch.from_numpy(np.ascontiguousarray(x).reshape(-1)).to(td))
    return flat, flat[: x.size].view(x.shape)


def run_prepad(ma, q, k, v, m, b, T, dtype, lens=None):
    import torch

    td = _td(dtype)
    if ma.path_name == "fused" and not ma.fused_applies(q.shape[-1], m, b, ma.dtype_code(td)):
        pytest.skip("the fused kernel covers 16-bit elements, d = 64, m and b <= 16")
    bufs = [_guarded(torch, x, td) for x in (q, k, v)]
    oflat, out = _guarded(torch, np.full(q.shape, np.nan, dtype=np.float32), td)
    tl = None if lens is None else torch.tensor(lens, dtype=torch.int32, device="cuda")
    ma.monarch_attn_fwd_prepad(bufs[0][1], bufs[1][1], bufs[2][1], out, m, b, T, lens=tl)
    torch.cuda.synchronize()
    assert bool(torch.isnan(oflat[q.size:]).all()), "a store past the last row"
    return out


CASES = [
    (2, 3, 197, 15, 14, 64, 2, "bf16"),     # ViT-B/16 with its class token at the front
    (1, 2, 10, 3, 4, 64, 2, "f32"),
    (1, 2, 33, 3, 16, 64, 3, "bf16"),
    (1, 2, 250, 16, 16, 64, 2, "f16"),
    (1, 1, 130, 2, 128, 64, 2, "bf16"),     # first block holds 2 real keys
    (2, 2, 1000, 8, 128, 64, 1, "f16"),
    (1, 1, 7600, 60, 128, 48, 2, "bf16"),   # GPS shape
    (1, 2, 250, 16, 16, 64, 2, "f32"),
    (1, 2, 5, 1, 16, 64, 2, "bf16"),        # one block: exact attention over the real keys
]


@pytest.mark.parametrize("B,H,n,m,b,d,T,dtype", CASES)
def test_prepad_matches_oracle(ma, B, H, n, m, b, d, T, dtype):
    if dtype == "f32" and (16 * -(-m // 16) * 64 > 8192 or 16 * -(-b // 16) * 64 > 8192):
        pytest.skip("fp32 tile exceeds the supported LDS budget")
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=n + 17 * b, scale=1.5)
    ref = oracle.monarch_attention_prepad(q, k, v, m, b, T)
    o = run_prepad(ma, q, k, v, m, b, T, dtype).double().cpu().numpy()
    assert np.isfinite(o).all()
    err = oracle.rel_frobenius(o, ref)
    # the classes of the pre-padded problem: row r sits at position m b - n + r
    shift = m * b - n
    ref_p = np.concatenate([np.zeros(ref.shape[:2] + (shift, d)), ref], axis=2)
    o_p = np.concatenate([np.zeros(o.shape[:2] + (shift, d)), o], axis=2)
    cls, where = parity.worst_class(o_p, ref_p, b)
    print(f"prepad {ma.path_name} {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T}: rel_frob={err:.3e} "
          f"max_class={cls:.3e} at {where}", flush=True)
    assert err <= TOL[dtype]
    assert cls <= parity.class_bar(TOL[dtype])


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("n,m,b,T", [(197, 15, 14, 2), (250, 16, 16, 3), (1000, 8, 128, 2), (37, 3, 13, 2)])
def test_prepad_is_reversed_postpad_bitwise(ma, dtype, n, m, b, T):
    import torch

    if dtype == "f32" and (16 * -(-m // 16) * 64 > 8192 or 16 * -(-b // 16) * 64 > 8192):
        pytest.skip("fp32 tile exceeds the supported LDS budget")
    q, k, v = si.random_qkv(2, 2, n, 64, dtype, seed=n, scale=1.5)
    got = run_prepad(ma, q, k, v, m, b, T, dtype)
    td = _td(dtype)
    rq, rk, rv = (torch.from_numpy(np.ascontiguousarray(x[:, :, ::-1])).to(td).cuda() for x in (q, k, v))
    post = torch.full_like(rq, float("nan"))
    ma.monarch_attn_fwd(rq, rk, rv, post, m, b, T)
    torch.cuda.synchronize()
    assert torch.equal(got, torch.flip(post, dims=[2]))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,m,b,T", [(96, 12, 8, 2), (384, 8, 48, 1), (197, 15, 14, 2), (16384, 128, 128, 2)])
def test_prepad_left_padded_batch(ma, dtype, n, m, b, T):
    """A left-padded batch: real rows last; the rows before them hold NaN on
    input and must come out as zero."""
    import torch

    if dtype == "f32" and (16 * -(-m // 16) * 64 > 8192 or 16 * -(-b // 16) * 64 > 8192):
        pytest.skip("fp32 tile exceeds the supported LDS budget")
    B = 5 if n < 4096 else 2
    lens = [n, 0, 1, min(n, b + 1), n // 3][:B]
    q, k, v = si.random_qkv(B, 1 if n >= 4096 else 2, n, 64, dtype, seed=n + b, scale=1.5)
    for bi, ln in enumerate(lens):
        for x in (q, k, v):
            x[bi, :, : n - ln] = np.nan
    o = run_prepad(ma, q, k, v, m, b, T, dtype, lens=lens).double().cpu().numpy()
    qz, kz, vz = (np.nan_to_num(x, nan=0.0) for x in (q, k, v))
    ref = oracle.monarch_attention_prepad(qz, kz, vz, m, b, T, lens=np.array(lens))
    assert np.isfinite(o).all()
    for bi, ln in enumerate(lens):
        assert np.all(o[bi, :, : n - ln] == 0.0)
    real = np.concatenate([o[bi, :, n - ln:].ravel() for bi, ln in enumerate(lens)])
    want = np.concatenate([ref[bi, :, n - ln:].ravel() for bi, ln in enumerate(lens)])
    err = float(np.linalg.norm(real - want) / np.linalg.norm(want))
    print(f"left-padded {ma.path_name} {dtype} N{n} m{m} b{b} T{T} lens={lens}: rel_frob={err:.3e}", flush=True)
    assert err <= TOL[dtype]


def test_grouped_path_refuses_prepad(lib):
    import torch

    prev = lib.monarch_attn_set_path(lib.PATH_GROUPED)
    try:
        q = torch.zeros(1, 1, 250, 64, device="cuda", dtype=torch.bfloat16)
        out = torch.full_like(q, 3.0)
        with pytest.raises(lib.MonarchAttnError) as exc:
            lib.monarch_attn_fwd_prepad(q, q.clone(), q.clone(), out, 16, 16, 2)
        assert exc.value.status == lib.MA_EUNSUPPORTED
        torch.cuda.synchronize()
        assert bool((out == 3.0).all())
    finally:
        lib.monarch_attn_set_path(prev)
