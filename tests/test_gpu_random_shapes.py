"""Seeded random shapes against the oracle: the forward pass on both paths,
padded batches, and the gradient.

Each case draws its own element type, m and b (1..128), N in ((m - 1) b, m b],
d (every multiple of 16 bytes up to 128), T, batch and head counts and the
input scale from its seed, and keeps only shapes the library reports as
supported (monarch_attn_check, no GPU call).  Bars as in the other parity
tests: rel-Frobenius <= 1e-5 / 2e-5 (fp32 forward / gradient) and <= 2e-2 /
3e-2 (bf16, fp16), outputs starting as NaN so that an unwritten element
fails, rows past a sequence's length exactly zero.  The forward outputs
also hold twice the bar on every (batch, head, residue class j) alone.
"""
import numpy as np
import pytest

import oracle
import oracle.backward as ob
import parity
import synth_inputs as si

pytestmark = pytest.mark.gpu

FWD_TOL = {"f32": 1e-5, "bf16": 2e-2, "f16": 2e-2}
BWD_TOL = {"f32": 2e-5, "bf16": 3e-2, "f16": 3e-2}


@pytest.fixture(scope="module")
def ma():
    import torch

    assert torch.cuda.is_available(), "no GPU visible"
    import paper_2505_18698_amd as lib

    return lib


def _td(dtype):
    import torch

    return {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]


def _code(ma, dtype):
    return {"f32": ma.MA_F32, "bf16": ma.MA_BF16, "f16": ma.MA_F16}[dtype]


def draw(ma, seed, max_np, max_t, check, max_mb=128, max_d=128, dtypes=("f32", "bf16", "f16"), min_mb=1):
    """(dtype, B, H, m, b, n, d, T, scale) for case `seed`: the first supported draw."""
    rs = np.random.RandomState(seed)
    while True:
        dtype = str(rs.choice(list(dtypes)))
        m, b = int(rs.randint(min_mb, max_mb + 1)), int(rs.randint(min_mb, max_mb + 1))
        if m * b > max_np:
            continue
        n = int(rs.randint((m - 1) * b + 1, m * b + 1))
        unit = 4 if dtype == "f32" else 8
        d = unit * int(rs.randint(1, max_d // unit + 1))
        T = int(rs.randint(1, max_t + 1))
        if check(n, d, m, b, T, _code(ma, dtype)) != 0:
            continue
        B, H = int(rs.randint(1, 3)), int(rs.randint(1, 3))
        scale = float(rs.choice([0.5, 1.0, 1.5]))
        return dtype, B, H, m, b, n, d, T, scale


def assert_classes(o, ref, b, dtype, label):
    cls, where = parity.worst_class(o, ref, b)
    print(f"  max_class={cls:.3e} at (batch, head, j)={where}", flush=True)
    assert cls <= parity.class_bar(FWD_TOL[dtype]), (label, cls, where)


def _to_dev(arrays, dtype):
    import torch

    return [torch.from_numpy(x).to(_td(dtype)).cuda() for x in arrays]


@pytest.mark.parametrize("path", ["auto", "half_steps"])
@pytest.mark.parametrize("case", range(100))
def test_random_forward(ma, case, path):
    import torch

    dtype, B, H, m, b, n, d, T, scale = draw(ma, 7000 + case, 4096, 6, ma.monarch_attn_check)
    label = f"fwd {path} {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T} scale{scale}"
    print(label, flush=True)
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=7000 + case, scale=scale)
    ref = oracle.monarch_attention(q, k, v, m, b, T)
    prev = ma.monarch_attn_set_path(ma.PATH_AUTO if path == "auto" else ma.PATH_HALF_STEPS)
    try:
        tq, tk, tv = _to_dev((q, k, v), dtype)
        out = torch.full_like(tq, float("nan"))
        ma.monarch_attn_fwd(tq, tk, tv, out, m, b, T)
        torch.cuda.synchronize()
    finally:
        ma.monarch_attn_set_path(prev)
    o = out.double().cpu().numpy()
    assert np.isfinite(o).all(), label
    err = oracle.rel_frobenius(o, ref)
    print(f"  rel_frob={err:.3e}", flush=True)
    assert err <= FWD_TOL[dtype], (label, err)
    assert_classes(o, ref, b, dtype, label)


@pytest.mark.parametrize("case", range(40))
def test_random_grouped(ma, case):
    """The grouped kernel's scope (16-bit, d <= 64, m <= 64, b <= 32) with
    head counts from 1 to 96, so that the group size and the number of
    resident rounds vary: parity with the oracle, and the bits of the
    half-step kernels."""
    import torch

    def check(n, d, m, b, T, code):
        return ma.monarch_attn_check(n, d, m, b, T, code) if b <= 32 else 1

    dtype, B, H, m, b, n, d, T, scale = draw(ma, 7800 + case, 2048, 4, check, max_mb=64, max_d=64,
                                              dtypes=("bf16", "f16"))
    H = int(np.random.RandomState(7800 + case).choice([1, 3, 16, 48]))
    label = f"grouped {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T}"
    print(label, flush=True)
    assert ma.grouped_applies(d, m, b, _code(ma, dtype))
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=7800 + case, scale=scale)
    ref = oracle.monarch_attention(q, k, v, m, b, T)
    outs = {}
    for path in (ma.PATH_GROUPED, ma.PATH_HALF_STEPS):
        prev = ma.monarch_attn_set_path(path)
        try:
            tq, tk, tv = _to_dev((q, k, v), dtype)
            out = torch.full_like(tq, float("nan"))
            ma.monarch_attn_fwd(tq, tk, tv, out, m, b, T)
            torch.cuda.synchronize()
        finally:
            ma.monarch_attn_set_path(prev)
        outs[path] = out.cpu()
    assert torch.equal(outs[ma.PATH_GROUPED], outs[ma.PATH_HALF_STEPS]), label
    o = outs[ma.PATH_GROUPED].double().numpy()
    assert np.isfinite(o).all(), label
    err = oracle.rel_frobenius(o, ref)
    print(f"  rel_frob={err:.3e}", flush=True)
    assert err <= FWD_TOL[dtype], (label, err)
    assert_classes(o, ref, b, dtype, label)


@pytest.mark.parametrize("case", range(40))
def test_random_small_heads(ma, case):
    """m, b <= 16 and d <= 64 in 16-bit types: the one-workgroup-per-head
    kernel (the automatic path), the grouped kernel and the half-step kernels."""
    import torch

    dtype, B, H, m, b, n, d, T, scale = draw(ma, 7500 + case, 256, 5, ma.monarch_attn_check, max_mb=16, max_d=64,
                                              dtypes=("bf16", "f16"))
    B, H = 2 * B, 3 * H  # several workgroups
    label = f"small {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T}"
    print(label, flush=True)
    assert ma.fused_applies(d, m, b, _code(ma, dtype))
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=7500 + case, scale=scale)
    ref = oracle.monarch_attention(q, k, v, m, b, T)
    for path in (ma.PATH_FUSED, ma.PATH_GROUPED, ma.PATH_HALF_STEPS):
        prev = ma.monarch_attn_set_path(path)
        try:
            tq, tk, tv = _to_dev((q, k, v), dtype)
            out = torch.full_like(tq, float("nan"))
            ma.monarch_attn_fwd(tq, tk, tv, out, m, b, T)
            torch.cuda.synchronize()
        finally:
            ma.monarch_attn_set_path(prev)
        o = out.double().cpu().numpy()
        assert np.isfinite(o).all(), (label, path)
        err = oracle.rel_frobenius(o, ref)
        print(f"  path {path} rel_frob={err:.3e}", flush=True)
        assert err <= FWD_TOL[dtype], (label, path, err)
        assert_classes(o, ref, b, dtype, (label, path))


@pytest.mark.parametrize("case", range(40))
def test_random_padded_batch(ma, case):
    import torch

    dtype, _, H, m, b, n, d, T, scale = draw(ma, 8000 + case, 4096, 3, ma.monarch_attn_check)
    rs = np.random.RandomState(8500 + case)
    B = int(rs.randint(2, 5))
    edges = [0, 1, n, max(0, n - 1), min(n, b), min(n, b + 1)]
    lens = [int(rs.choice(edges)) if rs.rand() < 0.4 else int(rs.randint(0, n + 1)) for _ in range(B)]
    label = f"varlen {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T} lens={lens}"
    print(label, flush=True)
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=8000 + case, scale=scale)
    ref = oracle.monarch_attention_varlen(q, k, v, np.array(lens), m, b, T)
    tq, tk, tv = _to_dev((q, k, v), dtype)
    out = torch.full_like(tq, float("nan"))
    ma.monarch_attn_fwd_varlen(tq, tk, tv, out, torch.tensor(lens, dtype=torch.int32, device="cuda"), m, b, T)
    torch.cuda.synchronize()
    o = out.double().cpu().numpy()
    assert np.isfinite(o).all(), label
    for bi, ln in enumerate(lens):
        assert np.all(o[bi, :, ln:] == 0.0), (label, bi)
    real = np.concatenate([o[bi, :, :ln].ravel() for bi, ln in enumerate(lens)])
    want = np.concatenate([ref[bi, :, :ln].ravel() for bi, ln in enumerate(lens)])
    err = float(np.linalg.norm(real - want) / np.linalg.norm(want)) if np.linalg.norm(want) > 0 else 0.0
    print(f"  rel_frob={err:.3e}", flush=True)
    assert err <= FWD_TOL[dtype], (label, err)


@pytest.mark.parametrize("case", range(48))
def test_random_gradient(ma, case):
    import torch

    dtype, B, H, m, b, n, d, T, scale = draw(ma, 9000 + case, 1024, 3, ma.LIB.monarch_attn_bwd_check)
    label = f"bwd {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T} scale{scale}"
    print(label, flush=True)
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=9000 + case, scale=scale)
    g = si.random_cotangent((B, H, n, d), dtype, seed=9000 + case)
    tq, tk, tv, tg = _to_dev((q, k, v, g), dtype)
    outs = [torch.full_like(tq, float("nan")) for _ in range(3)]
    ma.monarch_attn_bwd(tq, tk, tv, tg, *outs, m, b, T)
    torch.cuda.synchronize()
    got = [x.double().cpu().numpy() for x in outs]
    want = [np.zeros(q.shape) for _ in range(3)]
    for i in range(B):
        for h in range(H):
            for w, r in zip(want, ob.autograd_grads(q[i, h], k[i, h], v[i, h], g[i, h], m, b, T)):
                w[i, h] = r
    errs = []
    for name, x, w in zip(("dq", "dk", "dv"), got, want):
        assert np.isfinite(x).all(), (label, name)
        errs.append(oracle.rel_frobenius(x, w))
    unit = parity.worst_grad_unit(*got, *want, b)
    print(f"  rel_frob dq={errs[0]:.3e} dk={errs[1]:.3e} dv={errs[2]:.3e} max_unit={unit[0]:.3e} ({unit[1]} at {unit[2]})",
          flush=True)
    for name, e in zip(("dq", "dk", "dv"), errs):
        assert e <= BWD_TOL[dtype], (label, name, e)
    assert unit[0] <= parity.class_bar(BWD_TOL[dtype]), (label, unit)


# relative to max |f|; the derivation is beside the objective parity test
OBJ_TOL = {"f32": 1e-5, "bf16": 1e-3, "f16": 1e-3}


@pytest.mark.parametrize("case", range(30))
def test_random_objective(ma, case):
    import torch

    dtype, B, H, m, b, n, d, T, scale = draw(ma, 9500 + case, 4096, 4, ma.monarch_attn_check)
    label = f"objective {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T} scale{scale}"
    print(label, flush=True)
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=9500 + case, scale=scale)
    ref_o, ref_f = oracle.monarch_attention_objective(q, k, v, m, b, T)
    tq, tk, tv = _to_dev((q, k, v), dtype)
    out = torch.full_like(tq, float("nan"))
    obj = torch.full((B, H, T), float("nan"), dtype=torch.float32, device="cuda")
    ma.monarch_attn_fwd_objective(tq, tk, tv, out, obj, m, b, T)
    torch.cuda.synchronize()
    o, f = out.double().cpu().numpy(), obj.double().cpu().numpy()
    assert np.isfinite(o).all() and np.isfinite(f).all(), label
    err = oracle.rel_frobenius(o, ref_o)
    rel = float(np.abs(f - ref_f).max() / max(np.abs(ref_f).max(), 1e-30))
    print(f"  rel_frob={err:.3e} objective max rel err={rel:.3e}", flush=True)
    assert err <= FWD_TOL[dtype], (label, err)
    assert rel <= OBJ_TOL[dtype], (label, rel)
    assert_classes(o, ref_o, b, dtype, label)


def _lens(rs, B, n, b):
    edges = [0, 1, n, max(0, n - 1), min(n, b), min(n, b + 1)]
    return [int(rs.choice(edges)) if rs.rand() < 0.4 else int(rs.randint(0, n + 1)) for _ in range(B)]


@pytest.mark.parametrize("case", range(24))
def test_random_padded_batch_gradient(ma, case):
    """monarch_attn_bwd_varlen against the autograd oracle of each real
    sequence (reading 10b); rows past a length get exactly zero gradient."""
    import torch

    dtype, _, H, m, b, n, d, T, scale = draw(ma, 9700 + case, 1024, 3, ma.LIB.monarch_attn_bwd_check)
    rs = np.random.RandomState(9800 + case)
    B = int(rs.randint(2, 5))
    lens = _lens(rs, B, n, b)
    label = f"bwd varlen {dtype} B{B} H{H} N{n} m{m} b{b} d{d} T{T} lens={lens}"
    print(label, flush=True)
    q, k, v = si.random_qkv(B, H, n, d, dtype, seed=9700 + case, scale=scale)
    g = si.random_cotangent((B, H, n, d), dtype, seed=9700 + case)
    tq, tk, tv, tg = _to_dev((q, k, v, g), dtype)
    outs = [torch.full_like(tq, float("nan")) for _ in range(3)]
    ma.monarch_attn_bwd_varlen(tq, tk, tv, tg, *outs, torch.tensor(lens, dtype=torch.int32, device="cuda"), m, b, T)
    torch.cuda.synchronize()
    got = [x.double().cpu().numpy() for x in outs]
    have, want = [[], [], []], [[], [], []]
    full = [np.zeros(q.shape) for _ in range(3)]  # the references, zero past each length
    for bi, ln in enumerate(lens):
        for x in got:
            assert np.isfinite(x).all(), label
            assert np.all(x[bi, :, ln:] == 0.0), (label, bi)
        for h in range(H):
            ref = ob.autograd_grads(q[bi, h, :ln], k[bi, h, :ln], v[bi, h, :ln], g[bi, h, :ln], m, b, T,
                                    batch_padding=True)
            for c in range(3):
                want[c].append(ref[c].ravel())
                have[c].append(got[c][bi, h, :ln].ravel())
                full[c][bi, h, :ln] = ref[c]
    errs = [oracle.rel_frobenius(np.concatenate(x), np.concatenate(w)) if np.concatenate(w).size else 0.0
            for x, w in zip(have, want)]
    unit = parity.worst_grad_unit(*got, *full, b)
    print(f"  rel_frob dq={errs[0]:.3e} dk={errs[1]:.3e} dv={errs[2]:.3e} max_unit={unit[0]:.3e} ({unit[1]} at {unit[2]})",
          flush=True)
    for name, e in zip(("dq", "dk", "dv"), errs):
        assert e <= BWD_TOL[dtype], (label, name, e)
    assert unit[0] <= parity.class_bar(BWD_TOL[dtype]), (label, unit)


@pytest.mark.parametrize("case", range(12))
def test_random_long_sequences(ma, case):
    """m, b in 64..128 (N from 4033 to the headline's 16384), one batch element."""
    import torch

    dtype, _, H, m, b, n, d, T, scale = draw(ma, 9900 + case, 16384, 3, ma.monarch_attn_check, min_mb=64)
    label = f"long {dtype} H{H} N{n} m{m} b{b} d{d} T{T} scale{scale}"
    print(label, flush=True)
    q, k, v = si.random_qkv(1, H, n, d, dtype, seed=9900 + case, scale=scale)
    ref = oracle.monarch_attention(q, k, v, m, b, T)
    tq, tk, tv = _to_dev((q, k, v), dtype)
    out = torch.full_like(tq, float("nan"))
    ma.monarch_attn_fwd(tq, tk, tv, out, m, b, T)
    torch.cuda.synchronize()
    o = out.double().cpu().numpy()
    assert np.isfinite(o).all(), label
    err = oracle.rel_frobenius(o, ref)
    print(f"  rel_frob={err:.3e}", flush=True)
    assert err <= FWD_TOL[dtype], (label, err)
    assert_classes(o, ref, b, dtype, label)


def _max_t(ma, dtype, fp32_max, bwd=False):
    """The largest T the library takes for the element type."""
    return fp32_max if dtype == "f32" else ma.MAX_T_16BIT_BWD if bwd else ma.MAX_T_16BIT


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("path", ["auto", "half_steps"])
@pytest.mark.parametrize("m,b,d", [(16, 16, 64), (24, 40, 48)])
def test_maximum_step_count_forward(ma, dtype, path, m, b, d):
    """The largest T the forward takes for the element type (64 for fp32:
    128 half-step launches or one fused launch), with the objective after
    every step, at the fixed bars."""
    import torch

    T = _max_t(ma, dtype, 64)
    n = m * b - 3
    q, k, v = si.random_qkv(2, 2, n, d, dtype, seed=64 + m, scale=1.5)
    ref_o, ref_f = oracle.monarch_attention_objective(q, k, v, m, b, T)
    prev = ma.monarch_attn_set_path(ma.PATH_AUTO if path == "auto" else ma.PATH_HALF_STEPS)
    try:
        tq, tk, tv = _to_dev((q, k, v), dtype)
        out = torch.full_like(tq, float("nan"))
        ma.monarch_attn_fwd(tq, tk, tv, out, m, b, T)
        out2 = torch.full_like(tq, float("nan"))
        obj = torch.full((2, 2, T), float("nan"), dtype=torch.float32, device="cuda")
        ma.monarch_attn_fwd_objective(tq, tk, tv, out2, obj, m, b, T)
        torch.cuda.synchronize()
    finally:
        ma.monarch_attn_set_path(prev)
    o, o2, f = (x.double().cpu().numpy() for x in (out, out2, obj))
    assert torch.equal(out, out2)
    err = oracle.rel_frobenius(o, ref_o)
    rel = float(np.abs(f - ref_f).max() / np.abs(ref_f).max())
    label = f"T={T} {path} {dtype} m{m} b{b} d{d}"
    print(f"{label}: rel_frob={err:.3e} objective={rel:.3e}", flush=True)
    assert np.isfinite(o).all() and np.isfinite(f).all()
    assert err <= FWD_TOL[dtype] and rel <= OBJ_TOL[dtype], (label, err, rel)
    assert_classes(o, ref_o, b, dtype, label)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("T", [3, 4])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_ill_conditioned_class(ma, dtype, T, seed):
    """The random shape whose worst residue class is the most sensitive found
    (m = 59, b = 38, d = 112: the fp64 method moves that class by up to
    9.4e-2 at T = 4 under half an ulp of its bf16 inputs), at the largest
    16-bit step counts: every class within twice the whole-tensor bar."""
    import torch

    m, b, d = 59, 38, 112
    n = m * b - 7 * seed
    q, k, v = si.random_qkv(1, 2, n, d, dtype, seed=1000 + seed, scale=1.5)
    ref = oracle.monarch_attention(q, k, v, m, b, T)
    tq, tk, tv = _to_dev((q, k, v), dtype)
    out = torch.full_like(tq, float("nan"))
    ma.monarch_attn_fwd(tq, tk, tv, out, m, b, T)
    torch.cuda.synchronize()
    o = out.double().cpu().numpy()
    err = oracle.rel_frobenius(o, ref)
    label = f"ill-conditioned {dtype} T{T} seed{seed} N{n}"
    print(f"{label}: rel_frob={err:.3e}", flush=True)
    assert np.isfinite(o).all() and err <= FWD_TOL[dtype], (label, err)
    assert_classes(o, ref, b, dtype, label)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_maximum_step_count_gradient(ma, dtype):
    """The largest T the gradient takes for the element type (32 for fp32: 64
    recompute and 64 sweep launches), at the fixed bars."""
    import torch

    m, b, d = 8, 8, 32
    T = _max_t(ma, dtype, 32, bwd=True)
    n = m * b - 5
    q, k, v = si.random_qkv(1, 2, n, d, dtype, seed=32, scale=1.5)
    g = si.random_cotangent((1, 2, n, d), dtype, seed=32)
    tq, tk, tv, tg = _to_dev((q, k, v, g), dtype)
    outs = [torch.full_like(tq, float("nan")) for _ in range(3)]
    ma.monarch_attn_bwd(tq, tk, tv, tg, *outs, m, b, T)
    torch.cuda.synchronize()
    got = [x.double().cpu().numpy() for x in outs]
    want = [np.zeros(q.shape) for _ in range(3)]
    for h in range(2):
        for w, r in zip(want, ob.autograd_grads(q[0, h], k[0, h], v[0, h], g[0, h], m, b, T)):
            w[0, h] = r
    errs = [oracle.rel_frobenius(x, w) for x, w in zip(got, want)]
    unit = parity.worst_grad_unit(*got, *want, b)
    print(f"T={T} gradient {dtype}: rel_frob dq={errs[0]:.3e} dk={errs[1]:.3e} dv={errs[2]:.3e} "
          f"max_unit={unit[0]:.3e} ({unit[1]} at {unit[2]})", flush=True)
    for x in got:
        assert np.isfinite(x).all()
    for e in errs:
        assert e <= BWD_TOL[dtype], (dtype, T, errs)
    assert unit[0] <= parity.class_bar(BWD_TOL[dtype]), (dtype, T, unit)
