"""Host-side checks of the C ABI that need no GPU: the library loads, it
exports every function include/monarch_attn.h declares, and malformed or
unsupported arguments are rejected before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "monarch_attn.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(monarch_attn_\w+)\s*\(", text)))


def test_header_declarations_match_binding():
    import paper_2505_18698_amd as ma

    assert _declared_functions() == sorted(ma.EXPORTS)


def test_library_exports_every_declared_symbol():
    import paper_2505_18698_amd as ma

    lib = ctypes.CDLL(ma.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name


FAKE = 1 << 20  # an aligned non-null address that is never dereferenced: every case fails validation first


@pytest.mark.parametrize(
    "args,code",
    [
        # (q, k, v, out, B, H, N, d, m, b, T, dtype)
        ((0, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),           # null q
        ((FAKE, FAKE, FAKE, 0, 1, 1, 256, 64, 16, 16, 1, 1), 1),               # null out
        ((FAKE, FAKE, FAKE, 2 * FAKE, -1, 1, 256, 64, 16, 16, 1, 1), 1),       # B < 0
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 0, 64, 1, 16, 1, 1), 1),           # N = 0 needs m = 0
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 16, 64, 0, 16, 1, 1), 1),          # m = 0 needs N = 0
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 257, 64, 16, 16, 1, 1), 1),        # N > m b
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 240, 64, 16, 16, 1, 1), 1),        # m > ceil(N / b)
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 64, 16, 16, 0, 1), 1),        # T = 0
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 64, 16, 16, 1, 7), 1),        # bad dtype
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 64, 0, 16, 1, 1), 1),         # m = 0
        ((FAKE + 2, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),    # misaligned q
        ((FAKE, FAKE, FAKE, FAKE + 64, 1, 1, 256, 64, 16, 16, 1, 1), 1),       # out overlaps q
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 100, 16, 16, 1, 1), 2),       # d not a multiple of 8
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 136, 16, 16, 1, 1), 2),       # d > 128
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 6, 16, 16, 1, 0), 2),         # fp32 d not a multiple of 4
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 512, 64, 2, 256, 1, 1), 2),        # b > 128
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 64, 16, 16, 65, 1), 2),       # T > 64
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 16384, 128, 128, 128, 1, 0), 2),   # fp32 tile too big
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1 << 24, 1 << 24, 256, 64, 16, 16, 1, 1), 2),  # B H * 16 >= 2^31
        ((FAKE, FAKE, FAKE, 2 * FAKE, 1 << 40, 1 << 40, 256, 64, 16, 16, 1, 1), 2),  # B H overflows int64
    ],
)
def test_invalid_arguments_rejected_before_any_hip_call(args, code):
    import paper_2505_18698_amd as ma

    rc = ma.monarch_attn_fwd_raw(*args, None)
    assert rc == code, ma.monarch_attn_last_error()
    assert ma.monarch_attn_last_error() != ""


@pytest.mark.parametrize(
    "shape,ok",
    [
        ((256, 64, 16, 16, 1, 0), True),
        ((196, 64, 14, 14, 2, 1), True),
        ((1024, 64, 32, 32, 2, 1), True),
        ((4096, 64, 64, 64, 3, 1), True),
        ((16384, 64, 128, 128, 2, 1), True),
        ((16384, 128, 128, 128, 2, 1), True),
        ((16384, 128, 128, 128, 2, 2), True),
        ((384, 64, 16, 24, 1, 1), True),
        ((7, 64, 7, 1, 1, 1), True),
        ((8192, 64, 64, 128, 2, 0), True),
        ((16384, 128, 128, 128, 2, 0), False),
        ((197, 64, 15, 14, 2, 1), True),      # post-padded to 210 rows
        ((7600, 64, 60, 128, 2, 1), True),
        ((5, 64, 1, 16, 1, 1), True),
        ((196, 64, 15, 14, 2, 1), False),     # m != ceil(N / b)
        ((256, 72, 16, 16, 3, 1), True),      # DiT head dimension
        ((7600, 48, 60, 128, 2, 1), True),    # GPS head dimension
        ((256, 96, 16, 16, 2, 2), True),
        ((256, 36, 16, 16, 2, 0), True),      # fp32: multiples of 4
        ((256, 100, 16, 16, 2, 1), False),
        ((16384, 96, 128, 128, 2, 0), False), # fp32 tile too big at D = 96
        ((274, 88, 4, 75, 2, 0), False),      # fp32: b = 75 takes a 128-row tile, 128 x 96 > 8192
        ((2923, 84, 37, 80, 1, 0), False),    # fp32: the same at b = 80
        ((4096, 128, 64, 64, 2, 0), True),    # fp32: 64-row tiles at D = 128
        ((2560, 96, 40, 64, 2, 0), True),     # fp32: 64 x 96
    ],
)
def test_supported_shapes(shape, ok):
    import paper_2505_18698_amd as ma

    assert (ma.monarch_attn_check(*shape) == 0) == ok


@pytest.mark.parametrize("dtype", [1, 2])
def test_step_count_cap_of_16bit_types(dtype):
    """bf16 and fp16 take T up to the validated count (forward and gradient
    apart); fp32 up to 64 (32 for the gradient)."""
    import paper_2505_18698_amd as ma

    t16, t16b = ma.MAX_T_16BIT, ma.MAX_T_16BIT_BWD
    assert ma.monarch_attn_check(256, 64, 16, 16, t16, dtype) == 0
    assert ma.monarch_attn_check(256, 64, 16, 16, t16 + 1, dtype) == ma.MA_EUNSUPPORTED
    assert "validated" in ma.monarch_attn_last_error()
    assert ma.monarch_attn_bwd_check(256, 64, 16, 16, t16b, dtype) == 0
    assert ma.monarch_attn_bwd_check(256, 64, 16, 16, t16b + 1, dtype) == ma.MA_EUNSUPPORTED
    assert ma.monarch_attn_check(256, 64, 16, 16, 64, 0) == 0
    assert ma.monarch_attn_check(256, 64, 16, 16, 65, 0) == ma.MA_EUNSUPPORTED
    assert ma.monarch_attn_bwd_check(256, 64, 16, 16, 32, 0) == 0
    assert ma.monarch_attn_bwd_check(256, 64, 16, 16, 33, 0) == ma.MA_EUNSUPPORTED
    rc = ma.monarch_attn_fwd_raw(FAKE, FAKE, FAKE, 2 * FAKE, 1, 1, 256, 64, 16, 16, t16 + 1, dtype, None)
    assert rc == ma.MA_EUNSUPPORTED


def test_step_count_caps_match_the_header():
    import paper_2505_18698_amd as ma

    text = open(HEADER).read()
    assert re.search(r"#define MONARCH_ATTN_MAX_T_16BIT (\d+)", text).group(1) == str(ma.MAX_T_16BIT)
    assert re.search(r"#define MONARCH_ATTN_MAX_T_16BIT_BWD (\d+)", text).group(1) == str(ma.MAX_T_16BIT_BWD)


def test_build_id_matches_the_sources():
    """The library carries the hash of the sources it was built from, and it
    is that of the sources in the tree (the binding refuses it otherwise)."""
    import importlib.util

    import paper_2505_18698_amd as ma

    spec = importlib.util.spec_from_file_location("_b", os.path.join(ROOT, "paper_2505_18698_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert ma.monarch_attn_build_id() == mod.source_hash()
    assert re.fullmatch(r"[0-9a-f]{16}", ma.monarch_attn_build_id())


def test_workspace_bytes_formula():
    import paper_2505_18698_amd as ma

    B, H, N, d = 1, 16, 16384, 64
    got = ma.monarch_attn_workspace_bytes(B, H, N, d, 128, 128, 2, 1)
    state = B * H * N * d * 2   # alpha_R, alpha_L, Y
    cvec = B * H * N * 4        # c_R, c_L
    assert got == 3 * state + 2 * cvec
    assert ma.monarch_attn_workspace_bytes(B, H, N, d, 128, 128, 4, 1) == got  # independent of T
    assert ma.monarch_attn_workspace_bytes(B, H, N, d, 128, 127, 2, 1) == 0
    # a padded sequence: the states cover m * b rows
    padded = ma.monarch_attn_workspace_bytes(1, 1, 197, 64, 15, 14, 2, 1)
    assert padded == 3 * _align(210 * 64 * 2) + 2 * _align(210 * 4)
    # d = 72: state rows of 72 elements (the kernels' tiles are 96 wide; the padding never reaches memory)
    assert ma.monarch_attn_workspace_bytes(1, 2, 256, 72, 16, 16, 2, 1) == 3 * _align(2 * 256 * 72 * 2) + 2 * _align(2 * 256 * 4)
    assert ma.monarch_attn_workspace_bytes(1, 2, 7600, 48, 60, 128, 2, 1) == 3 * _align(2 * 7680 * 48 * 2) + 2 * _align(2 * 7680 * 4)


def _align(x):
    return (x + 255) // 256 * 256


def test_fused_path_applicability():
    import paper_2505_18698_amd as ma

    assert ma.fused_applies(64, 14, 14, ma.MA_BF16)
    assert ma.fused_applies(64, 16, 16, ma.MA_F16)
    assert ma.fused_applies(64, 1, 16, ma.MA_BF16)
    assert not ma.fused_applies(64, 16, 17, ma.MA_BF16)
    assert not ma.fused_applies(128, 16, 16, ma.MA_BF16)
    assert not ma.fused_applies(64, 16, 16, ma.MA_F32)


def test_grouped_path_applicability():
    """The binding's mirror of the grouped kernel's scope (the C side is
    checked in the host-code sanitizer run)."""
    import paper_2505_18698_amd as ma

    assert ma.grouped_applies(64, 32, 32, ma.MA_BF16)
    assert ma.grouped_applies(64, 64, 32, ma.MA_F16)
    assert ma.grouped_applies(48, 1, 1, ma.MA_BF16)
    assert not ma.grouped_applies(64, 16, 33, ma.MA_BF16)
    assert not ma.grouped_applies(64, 65, 32, ma.MA_BF16)
    assert not ma.grouped_applies(72, 16, 16, ma.MA_BF16)
    assert not ma.grouped_applies(64, 16, 16, ma.MA_F32)


def test_timing_read_without_a_timed_call_fails_cleanly():
    import paper_2505_18698_amd as ma

    with pytest.raises(ma.MonarchAttnError):
        ma.monarch_attn_timing_read()


def test_set_path_rejects_unknown_values_and_returns_previous():
    import paper_2505_18698_amd as ma

    prev = ma.monarch_attn_set_path(ma.PATH_HALF_STEPS)
    assert ma.monarch_attn_set_path(prev) == ma.PATH_HALF_STEPS
    with pytest.raises(ma.MonarchAttnError):
        ma.monarch_attn_set_path(7)


def test_objective_rejects_null_obj():
    import paper_2505_18698_amd as ma

    rc = ma.LIB.monarch_attn_fwd_objective(FAKE, FAKE, FAKE, 2 * FAKE, None, 1, 1, 256, 64, 16, 16, 1, 1, None)
    assert rc == ma.MA_EINVAL
    assert "objective" in ma.monarch_attn_last_error()


def test_varlen_rejects_null_or_misaligned_lens():
    import paper_2505_18698_amd as ma

    f = ma.LIB.monarch_attn_fwd_varlen
    assert f(FAKE, FAKE, FAKE, 2 * FAKE, None, 2, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_EINVAL
    assert "lens" in ma.monarch_attn_last_error()
    assert f(FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE + 2, 2, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_EINVAL
    assert "aligned" in ma.monarch_attn_last_error()
    # lens inside out (written by the kernels while lens is read)
    assert f(FAKE, FAKE, FAKE, 2 * FAKE, 2 * FAKE + 64, 2, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_EINVAL
    assert "overlap" in ma.monarch_attn_last_error()
    # the shape checks of the plain call apply
    assert f(FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 2, 1, 256, 64, 15, 16, 1, 1, None) == ma.MA_EINVAL
    assert f(None, None, None, None, None, 0, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_OK


def test_bwd_varlen_rejects_null_or_misaligned_lens():
    import paper_2505_18698_amd as ma

    f = ma.LIB.monarch_attn_bwd_varlen
    t = [FAKE * (i + 1) for i in range(7)]  # q, k, v, dout, dq, dk, dv: 1 MiB apart, no overlap
    assert f(*t, None, 2, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_EINVAL
    assert "lens" in ma.monarch_attn_last_error()
    assert f(*t, 9 * FAKE + 2, 2, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_EINVAL
    assert "aligned" in ma.monarch_attn_last_error()
    assert f(*t, 5 * FAKE + 64, 2, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_EINVAL  # inside dq
    assert "overlap" in ma.monarch_attn_last_error()
    assert f(None, None, None, None, None, None, None, None, 0, 1, 256, 64, 16, 16, 1, 1, None) == ma.MA_OK
    assert f(*t, 9 * FAKE, 2, 1, 256, 64, 16, 16, 33, 1, None) == ma.MA_EUNSUPPORTED  # T > 32, as the plain call


# ---- the gradient entry point ----

@pytest.mark.parametrize(
    "args,code",
    [
        # (q, k, v, dout, dq, dk, dv, B, H, N, d, m, b, T, dtype)
        ((FAKE, FAKE, FAKE, FAKE, 0, 3 * FAKE, 4 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),           # null dq
        ((FAKE, FAKE, FAKE, 0, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),       # null dout
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1, -2, 256, 64, 16, 16, 1, 1), 1),   # H < 0
        ((FAKE, FAKE, FAKE, FAKE, FAKE + 64, 3 * FAKE, 4 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),   # dq overlaps q
        ((FAKE, FAKE, FAKE, 5 * FAKE, 2 * FAKE, 3 * FAKE, 5 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),  # dv overlaps dout
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 2 * FAKE + 64, 4 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),  # dk overlaps dq
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE + 8, 3 * FAKE, 4 * FAKE, 1, 1, 256, 64, 16, 16, 1, 1), 1),  # misaligned dq
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1, 1, 257, 64, 16, 16, 1, 1), 1),    # N > m b
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1, 1, 16512, 64, 129, 128, 1, 1), 2),  # m > 128
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1, 1, 16512, 64, 128, 129, 1, 1), 2),  # b > 128
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1, 1, 8192, 128, 128, 64, 1, 0), 2),  # fp32 m > 64, d > 96
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1, 1, 256, 64, 16, 16, 33, 1), 2),   # T > 32
        ((FAKE, FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 1 << 40, 1 << 40, 256, 64, 16, 16, 1, 1), 2),  # B H overflows
    ],
)
def test_bwd_invalid_arguments_rejected_before_any_hip_call(args, code):
    import paper_2505_18698_amd as ma

    rc = ma.LIB.monarch_attn_bwd(*args, None)
    assert rc == code, ma.monarch_attn_last_error()
    assert ma.monarch_attn_last_error() != ""


@pytest.mark.parametrize(
    "shape,ok",
    [
        ((256, 64, 16, 16, 1, 1), True),
        ((196, 64, 14, 14, 3, 1), True),
        ((197, 64, 15, 14, 2, 2), True),
        ((4096, 64, 64, 64, 2, 0), True),
        ((7, 8, 7, 1, 1, 1), True),
        ((1024, 64, 32, 32, 32, 0), True),
        ((1024, 64, 32, 32, 33, 0), False),
        ((1024, 64, 32, 32, 4, 1), True),
        ((1024, 64, 32, 32, 5, 1), False),       # bf16 gradient: T above its validated count
        ((16384, 64, 128, 128, 2, 1), True),
        ((8192, 64, 128, 64, 2, 1), True),
        ((384, 64, 3, 128, 1, 1), True),
        ((7600, 48, 60, 128, 2, 1), True),
        ((16384, 64, 128, 128, 2, 0), True),
        ((16384, 128, 128, 128, 2, 1), True),    # 128-row tiles at d = 128 (16-bit unit tiles)
        ((8192, 128, 64, 128, 2, 1), True),
        ((8192, 128, 128, 64, 2, 2), True),
        ((8192, 128, 128, 64, 2, 0), False),     # fp32: the forward takes no 128-row block at d = 128
        ((256, 72, 16, 16, 3, 1), True),          # DiT
        ((256, 96, 16, 16, 2, 1), True),
        ((4096, 128, 64, 64, 2, 1), True),
        ((8192, 96, 128, 64, 2, 1), True),
        ((4096, 128, 64, 64, 2, 0), True),        # fp32 at the largest fp32 tile
        ((196, 64, 15, 14, 2, 1), False),
    ],
)
def test_bwd_supported_shapes(shape, ok):
    import paper_2505_18698_amd as ma

    assert (ma.monarch_attn_bwd_check(*shape) == 0) == ok


def test_bwd_workspace_bytes_formula():
    import paper_2505_18698_amd as ma

    B, H, N, d, m, b, T = 2, 3, 197, 64, 15, 14, 3
    Np, BH = m * b, B * H
    st, cs = _align(BH * Np * 64 * 2), _align(BH * Np * 4)
    acc, sg = _align(BH * N * d * 4), _align(BH * Np * 64 * 4)
    want = 2 * T * st + (2 * T - 1) * cs + 2 * acc + 3 * sg + 2 * cs
    assert ma.monarch_attn_bwd_workspace_bytes(B, H, N, d, m, b, T, ma.MA_BF16) == want
    # fp32 states are twice as wide; unsupported shapes give 0
    st32 = _align(BH * Np * 64 * 4)
    assert ma.monarch_attn_bwd_workspace_bytes(B, H, N, d, m, b, T, ma.MA_F32) == want + 2 * T * (st32 - st)
    assert ma.monarch_attn_bwd_workspace_bytes(1, 1, 16384, 128, 128, 128, 2, ma.MA_F32) == 0
    assert ma.monarch_attn_bwd_workspace_bytes(1, 1, 256, 64, 16, 16, 33, ma.MA_BF16) == 0
    # d = 72: states with rows of 72 elements, state gradients 96 wide
    B, H, N, d, m, b, T = 1, 2, 256, 72, 16, 16, 3
    Np, BH = m * b, B * H
    st, cs = _align(BH * Np * 72 * 2), _align(BH * Np * 4)
    acc, sg = _align(BH * N * d * 4), _align(BH * Np * 96 * 4)
    assert ma.monarch_attn_bwd_workspace_bytes(B, H, N, d, m, b, T, ma.MA_BF16) == \
        2 * T * st + (2 * T - 1) * cs + 2 * acc + 3 * sg + 2 * cs


@pytest.mark.parametrize("B,H,N,m", [(0, 4, 256, 16), (2, 0, 256, 16), (2, 4, 0, 0)])
def test_empty_calls_succeed_without_touching_pointers(B, H, N, m):
    """Nothing to compute: every entry point returns MA_OK with NULL pointers
    and launches nothing (no GPU is needed to run this)."""
    import paper_2505_18698_amd as ma

    assert ma.monarch_attn_fwd_raw(0, 0, 0, 0, B, H, N, 64, m, 16, 2, 1, None) == ma.MA_OK
    assert ma.LIB.monarch_attn_fwd_objective(None, None, None, None, None, B, H, N, 64, m, 16, 2, 1, None) == ma.MA_OK
    assert ma.LIB.monarch_attn_bwd(None, None, None, None, None, None, None, B, H, N, 64, m, 16, 2, 1, None) == ma.MA_OK
    assert ma.LIB.monarch_attn_exact_fwd(None, None, None, None, None, B, H, N, 64, 1, None) == ma.MA_OK
    # the other arguments are still checked
    assert ma.monarch_attn_fwd_raw(0, 0, 0, 0, B, H, N, 64, m, 16, 2, 9, None) == ma.MA_EINVAL
    assert ma.monarch_attn_fwd_raw(0, 0, 0, 0, B, H, N, 100, m, 16, 2, 1, None) == ma.MA_EUNSUPPORTED


def test_head_counts_that_overflow_a_grid_are_rejected():
    """B * H is checked without forming a product that could overflow."""
    import paper_2505_18698_amd as ma

    big = 1 << 40
    assert ma.LIB.monarch_attn_exact_fwd(FAKE, FAKE, FAKE, 2 * FAKE, None, big, big, 256, 64, 1, None) == \
        ma.MA_EUNSUPPORTED
    assert ma.LIB.monarch_attn_fwd_objective(FAKE, FAKE, FAKE, 2 * FAKE, 3 * FAKE, big, 3, 256, 64, 16, 16, 2, 1,
                                             None) == ma.MA_EUNSUPPORTED
    assert "too many heads" in ma.monarch_attn_last_error()
