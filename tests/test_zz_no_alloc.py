"""monarch_attn_fwd_noalloc through the C ABI against monarch_attn_fwd.

The entry point runs the same kernels with the states in the library's
per-device scratch array instead of the per-stream workspace, so its output
must equal monarch_attn_fwd's bit for bit.  Two calls in a row, the second
smaller, check that the array's leftover contents from the first call do not
leak into the second; a call whose states exceed the array is refused with
MA_EUNSUPPORTED and leaves `out` untouched.
"""
import ctypes

import numpy as np
import pytest

import synth_inputs as si

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ma():
    import torch

    assert torch.cuda.is_available(), "no GPU visible"
    import paper_2505_18698_amd as lib

    return lib


def _dev(torch, arrays, dtype):
    td = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    return [torch.from_numpy(x).to(td).cuda() for x in arrays]


def _raw_noalloc(ma, q, k, v, out, m, b, T, stream):
    B, H, N, d = q.shape
    return ma.LIB.monarch_attn_fwd_noalloc(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                                           ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                           B, H, N, d, m, b, T, ma.dtype_code(q.dtype), ctypes.c_void_p(stream))


def _pair(ma, torch, shape, dtype, seed):
    """(noalloc output, plain output) of one call of `shape` = (B, H, n, d, m, b, T)."""
    B, H, n, d, m, b, T = shape
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=seed, scale=1.5)
    tq, tk, tv = _dev(torch, (q, k, v), dtype)
    stream = torch.cuda.current_stream().cuda_stream
    got = torch.full_like(tq, float("nan"))
    rc = _raw_noalloc(ma, tq, tk, tv, got, m, b, T, stream)
    assert rc == ma.MA_OK, ma.monarch_attn_last_error()
    want = torch.full_like(tq, float("nan"))
    ma.monarch_attn_fwd(tq, tk, tv, want, m, b, T)
    torch.cuda.synchronize()
    return got, want


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize(
    "first,second",
    [
        ((1, 16, 4096, 64, 64, 64, 2), (1, 4, 1024, 64, 32, 32, 3)),      # 4K, then RoBERTa-sized heads
        ((2, 3, 2000, 64, 40, 50, 2), (1, 2, 197, 64, 15, 14, 1)),        # padded, then ViT with its class token
        ((1, 2, 8192, 64, 128, 64, 1), (2, 2, 300, 32, 19, 16, 2)),       # rectangular, then a smaller padded call
    ],
)
def test_noalloc_matches_fwd_twice(ma, dtype, first, second):
    import torch

    if dtype == "f32":
        first = first[:3] + (32,) + first[4:]
    for i, shape in enumerate((first, second)):
        got, want = _pair(ma, torch, shape, dtype, seed=17 + i)
        print(f"noalloc call {i + 1} {dtype} {shape}", flush=True)
        assert bool(torch.isfinite(got).all())
        assert torch.equal(got, want), float((got.float() - want.float()).abs().max())


def test_noalloc_fused_path_and_empty_call(ma):
    """Small heads take the one-workgroup-per-head kernel, which keeps its
    states in LDS; an empty call returns at once."""
    import torch

    got, want = _pair(ma, torch, (8, 12, 196, 64, 14, 14, 2), "bf16", seed=5)
    assert torch.equal(got, want)
    q = torch.empty((0, 4, 256, 64), device="cuda", dtype=torch.bfloat16)
    assert _raw_noalloc(ma, q, q, q, q, 16, 16, 2, 0) == ma.MA_OK


def test_noalloc_rejects_states_beyond_the_scratch(ma):
    import torch

    # 16 heads of 16384 rows at d = 64 in bf16: 3 x 32 MiB of states + c_R, c_L > 64 MiB
    B, H, n, d, m, b, T = 1, 16, 16384, 64, 128, 128, 2
    need = ma.monarch_attn_workspace_bytes(B, H, n, d, m, b, T, ma.MA_BF16)
    assert need > ma.NOALLOC_SCRATCH_BYTES
    tq = torch.zeros((B, H, n, d), device="cuda", dtype=torch.bfloat16)
    out = torch.full_like(tq, 3.0)
    rc = _raw_noalloc(ma, tq, tq, tq, out, m, b, T, torch.cuda.current_stream().cuda_stream)
    assert rc == ma.MA_EUNSUPPORTED
    assert "scratch" in ma.monarch_attn_last_error()
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())
    # the largest 4K call that fits runs
    got, want = _pair(ma, torch, (1, 32, 4096, 64, 64, 64, 1), "bf16", seed=9)
    assert ma.monarch_attn_workspace_bytes(1, 32, 4096, 64, 64, 64, 1, ma.MA_BF16) <= ma.NOALLOC_SCRATCH_BYTES
    assert torch.equal(got, want)
