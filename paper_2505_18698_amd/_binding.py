"""ctypes binding of libmonarch_attn.so: argument marshalling only.

Every step of the forward pass runs in the library's HIP kernels.  There is
no fallback: if the library is missing the import of this module fails.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmonarch_attn.so")

MA_F32, MA_BF16, MA_F16 = 0, 1, 2
MA_OK, MA_EINVAL, MA_EUNSUPPORTED, MA_EHIP, MA_ENOMEM = 0, 1, 2, 3, 4
STATUS_NAMES = {0: "MA_OK", 1: "MA_EINVAL", 2: "MA_EUNSUPPORTED", 3: "MA_EHIP", 4: "MA_ENOMEM"}
KIND_NAMES = {0: "r_half_step", 1: "l_half_step", 2: "r_half_step_final", 3: "monarch_apply",
              4: "monarch_fused_head", 5: "objective_sum", 6: "exact_attention", 7: "l_bwd", 8: "r_bwd",
              9: "monarch_fused_group"}
PATH_AUTO, PATH_HALF_STEPS, PATH_FUSED, PATH_GROUPED = 0, 1, 2, 3

# Every symbol declared in include/monarch_attn.h.
EXPORTS = (
    "monarch_attn_fwd",
    "monarch_attn_fwd_varlen",
    "monarch_attn_fwd_objective",
    "monarch_attn_exact_fwd",
    "monarch_attn_bwd",
    "monarch_attn_bwd_varlen",
    "monarch_attn_bwd_check",
    "monarch_attn_bwd_workspace_bytes",
    "monarch_attn_last_error",
    "monarch_attn_check",
    "monarch_attn_workspace_bytes",
    "monarch_attn_release_workspace",
    "monarch_attn_set_path",
    "monarch_attn_timing_enable",
    "monarch_attn_timing_read",
    "monarch_attn_build_id",
    "monarch_attn_fwd_noalloc",
    "monarch_attn_fwd_prepad",
)


class MonarchAttnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2505_18698_amd.build` "
            "(the HIP library is required, there is no fallback path)")
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    lib.monarch_attn_fwd.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, i32, vp]
    lib.monarch_attn_fwd.restype = ctypes.c_int
    lib.monarch_attn_fwd_varlen.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, i32, vp]
    lib.monarch_attn_fwd_varlen.restype = ctypes.c_int
    lib.monarch_attn_fwd_objective.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, i32, vp]
    lib.monarch_attn_fwd_objective.restype = ctypes.c_int
    lib.monarch_attn_exact_fwd.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i32, vp]
    lib.monarch_attn_exact_fwd.restype = ctypes.c_int
    lib.monarch_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, i32, vp]
    lib.monarch_attn_bwd.restype = ctypes.c_int
    lib.monarch_attn_bwd_varlen.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, i32, vp]
    lib.monarch_attn_bwd_varlen.restype = ctypes.c_int
    lib.monarch_attn_bwd_check.argtypes = [i64, i64, i64, i64, i32, i32]
    lib.monarch_attn_bwd_check.restype = ctypes.c_int
    lib.monarch_attn_bwd_workspace_bytes.argtypes = [i64, i64, i64, i64, i64, i64, i32, i32]
    lib.monarch_attn_bwd_workspace_bytes.restype = ctypes.c_size_t
    lib.monarch_attn_last_error.argtypes = []
    lib.monarch_attn_last_error.restype = ctypes.c_char_p
    lib.monarch_attn_check.argtypes = [i64, i64, i64, i64, i32, i32]
    lib.monarch_attn_check.restype = ctypes.c_int
    lib.monarch_attn_workspace_bytes.argtypes = [i64, i64, i64, i64, i64, i64, i32, i32]
    lib.monarch_attn_workspace_bytes.restype = ctypes.c_size_t
    lib.monarch_attn_release_workspace.argtypes = []
    lib.monarch_attn_release_workspace.restype = ctypes.c_int
    lib.monarch_attn_set_path.argtypes = [i32]
    lib.monarch_attn_set_path.restype = ctypes.c_int
    lib.monarch_attn_timing_enable.argtypes = [i32]
    lib.monarch_attn_timing_enable.restype = ctypes.c_int
    lib.monarch_attn_timing_read.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_int32), i32]
    lib.monarch_attn_timing_read.restype = ctypes.c_int32
    lib.monarch_attn_fwd_prepad.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, i32, vp]
    lib.monarch_attn_fwd_prepad.restype = ctypes.c_int
    lib.monarch_attn_fwd_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, i32, vp]
    lib.monarch_attn_fwd_noalloc.restype = ctypes.c_int
    lib.monarch_attn_build_id.argtypes = []
    lib.monarch_attn_build_id.restype = ctypes.c_char_p
    _check_provenance(lib)
    return lib


def _source_hash() -> str:
    import importlib.util

    spec = importlib.util.spec_from_file_location("_ma_build_hash", os.path.join(_PKG, "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod.source_hash()


def _check_provenance(lib) -> None:
    """Refuse a library built from other sources than the ones beside it."""
    built = lib.monarch_attn_build_id().decode()
    here = _source_hash()
    if built != here:
        raise ImportError(
            f"{LIB_PATH} was built from sources {built}, but the sources here hash to {here}: "
            "rebuild it (`python -m paper_2505_18698_amd.build`)")


def monarch_attn_build_id() -> str:
    """The source hash compiled into the library."""
    return LIB.monarch_attn_build_id().decode()


LIB = _load()
MAX_T_16BIT = 4      # MONARCH_ATTN_MAX_T_16BIT
MAX_T_16BIT_BWD = 4  # MONARCH_ATTN_MAX_T_16BIT_BWD


def monarch_attn_last_error() -> str:
    return LIB.monarch_attn_last_error().decode()


def _check(rc: int) -> None:
    if rc != MA_OK:
        raise MonarchAttnError(rc, monarch_attn_last_error())


def monarch_attn_fwd_raw(q: int, k: int, v: int, out: int, B: int, H: int, N: int, d: int,
                         m: int, b: int, T: int, dtype: int, stream: int | None) -> int:
    """The C call with integer device addresses; returns the status code."""
    return LIB.monarch_attn_fwd(q, k, v, out, B, H, N, d, m, b, T, dtype, stream or None)


def dtype_code(torch_dtype) -> int:
    import torch

    codes = {torch.float32: MA_F32, torch.bfloat16: MA_BF16, torch.float16: MA_F16}
    if torch_dtype not in codes:
        raise TypeError(f"unsupported dtype {torch_dtype}")
    return codes[torch_dtype]


def _check_tensors(q, k, v, out):
    import torch

    for name, t in (("q", q), ("k", k), ("v", v), ("out", out)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise TypeError(f"{name} must be a device tensor")
        if t.dim() != 4 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous [B, H, N, d] tensor")
        if t.shape != q.shape or t.dtype != q.dtype or t.device != q.device:
            raise ValueError(f"{name} must match q in shape, dtype and device")


def _stream(q, stream):
    """The hipStream_t to launch on: `stream`, or torch's current stream of
    q's device (read through torch's raw-stream hook where it exists: a
    fraction of the cost of torch.cuda.current_stream)."""
    import torch

    if stream is None:
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        if raw is not None:
            return raw(q.device.index)
        return torch.cuda.current_stream(q.device).cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


class _OnDevice:
    """Make q's device current for the call (a no-op when it already is)."""

    __slots__ = ("dev", "guard")

    def __init__(self, q):
        import torch

        self.dev = q.device.index
        self.guard = None if self.dev == torch.cuda.current_device() else torch.cuda.device(self.dev)

    def __enter__(self):
        if self.guard is not None:
            self.guard.__enter__()

    def __exit__(self, *exc):
        if self.guard is not None:
            return self.guard.__exit__(*exc)
        return False


def monarch_attn_fwd(q, k, v, out, m: int, b: int, T: int, stream=None):
    """O = MonarchAttention(q, k, v) into `out`; torch device tensors [B, H, N, d].

    `stream`: a torch.cuda.Stream, an integer hipStream_t, or None for torch's
    current stream.  Asynchronous on that stream.  Returns `out`.
    """
    import torch

    _check_tensors(q, k, v, out)
    B, H, N, d = q.shape
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(monarch_attn_fwd_raw(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                    B, H, N, d, m, b, T, dtype_code(q.dtype), stream))
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20  # MONARCH_ATTN_NOALLOC_SCRATCH_BYTES


def monarch_attn_fwd_noalloc(q, k, v, out, m: int, b: int, T: int, stream=None):
    """monarch_attn_fwd without any device allocation: the states go to the
    library's per-device scratch array (NOALLOC_SCRATCH_BYTES; larger calls
    raise MA_EUNSUPPORTED).  Calls that can overlap on one device race on that
    array.  Returns `out`."""
    _check_tensors(q, k, v, out)
    B, H, N, d = q.shape
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(LIB.monarch_attn_fwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                            B, H, N, d, m, b, T, dtype_code(q.dtype), stream))
    return out


def _check_lens(q, lens):
    import torch

    if not isinstance(lens, torch.Tensor) or lens.device != q.device or lens.dtype != torch.int32 \
            or not lens.is_contiguous() or tuple(lens.shape) != (q.shape[0],):
        raise ValueError("lens must be a contiguous int32 tensor [B] on the device of q")


def monarch_attn_fwd_varlen(q, k, v, out, lens, m: int, b: int, T: int, stream=None):
    """monarch_attn_fwd over a batch of post-padded sequences: lens (int32 device
    tensor [B]) holds the real rows of each batch element; rows >= lens[beta]
    of q, k, v count as zero whatever they hold, and those of out are written
    as zero.  Returns `out`."""
    import torch

    _check_tensors(q, k, v, out)
    _check_lens(q, lens)
    B, H, N, d = q.shape
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(LIB.monarch_attn_fwd_varlen(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                           lens.data_ptr(), B, H, N, d, m, b, T, dtype_code(q.dtype), stream))
    return out


def monarch_attn_fwd_prepad(q, k, v, out, m: int, b: int, T: int, lens=None, stream=None):
    """monarch_attn_fwd over pre-padded sequences (the padding rows first).
    lens None: all N rows real, pre-padded to m*b.  lens (int32 device tensor
    [B]): batch element beta's real rows are its LAST lens[beta] rows; its
    other rows of q, k, v count as zero and are written as zero in `out`.
    Returns `out`."""
    _check_tensors(q, k, v, out)
    if lens is not None:
        _check_lens(q, lens)
    B, H, N, d = q.shape
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(LIB.monarch_attn_fwd_prepad(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                           None if lens is None else lens.data_ptr(), B, H, N, d, m, b, T,
                                           dtype_code(q.dtype), stream))
    return out


def monarch_attn_fwd_objective(q, k, v, out, obj, m: int, b: int, T: int, stream=None):
    """monarch_attn_fwd, plus obj[B, H, T] (float32 device tensor): the variational
    objective f(M^(t); Q, K) after every step t.  Returns (out, obj)."""
    import torch

    _check_tensors(q, k, v, out)
    if not isinstance(obj, torch.Tensor) or obj.device != q.device or obj.dtype != torch.float32 \
            or not obj.is_contiguous() or tuple(obj.shape) != (q.shape[0], q.shape[1], T):
        raise ValueError("obj must be a contiguous float32 tensor [B, H, T] on the device of q")
    B, H, N, d = q.shape
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(LIB.monarch_attn_fwd_objective(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                              obj.data_ptr(), B, H, N, d, m, b, T, dtype_code(q.dtype), stream))
    return out, obj


def monarch_attn_exact_fwd(q, k, v, out, lse=None, stream=None):
    """Exact softmax attention into `out`; with `lse` (float32 device tensor
    [B, H, N]) also every row's logsumexp.  Returns (out, lse)."""
    import torch

    _check_tensors(q, k, v, out)
    B, H, N, d = q.shape
    if lse is not None and (not isinstance(lse, torch.Tensor) or lse.device != q.device
                            or lse.dtype != torch.float32 or not lse.is_contiguous()
                            or tuple(lse.shape) != (B, H, N)):
        raise ValueError("lse must be a contiguous float32 tensor [B, H, N] on the device of q")
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(LIB.monarch_attn_exact_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                          None if lse is None else lse.data_ptr(), B, H, N, d,
                                          dtype_code(q.dtype), stream))
    return out, lse


def monarch_attn_bwd(q, k, v, dout, dq, dk, dv, m: int, b: int, T: int, stream=None):
    """dq, dk, dv = the gradient of <MonarchAttention(q, k, v), dout> into the
    given tensors (all [B, H, N, d], one dtype).  Asynchronous on `stream`
    (torch's current stream when None).  Returns (dq, dk, dv)."""
    import torch

    _check_tensors(q, k, v, dout)
    _check_tensors(q, dq, dk, dv)
    B, H, N, d = q.shape
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(LIB.monarch_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(), dq.data_ptr(),
                                    dk.data_ptr(), dv.data_ptr(), B, H, N, d, m, b, T, dtype_code(q.dtype), stream))
    return dq, dk, dv


def monarch_attn_bwd_varlen(q, k, v, dout, dq, dk, dv, lens, m: int, b: int, T: int, stream=None):
    """The gradient of monarch_attn_fwd_varlen (lens: int32 device tensor [B]);
    rows >= lens[beta] of dq, dk, dv are written as zero.  Returns (dq, dk, dv)."""
    import torch

    _check_tensors(q, k, v, dout)
    _check_tensors(q, dq, dk, dv)
    _check_lens(q, lens)
    B, H, N, d = q.shape
    stream = _stream(q, stream)
    with _OnDevice(q):
        _check(LIB.monarch_attn_bwd_varlen(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(), dq.data_ptr(),
                                           dk.data_ptr(), dv.data_ptr(), lens.data_ptr(), B, H, N, d, m, b, T,
                                           dtype_code(q.dtype), stream))
    return dq, dk, dv


def monarch_attn_bwd_check(N: int, d: int, m: int, b: int, T: int, dtype: int) -> int:
    return LIB.monarch_attn_bwd_check(N, d, m, b, T, dtype)


def monarch_attn_bwd_workspace_bytes(B, H, N, d, m, b, T, dtype) -> int:
    return int(LIB.monarch_attn_bwd_workspace_bytes(B, H, N, d, m, b, T, dtype))


def monarch_attention(q, k, v, m: int, b: int, T: int, stream=None):
    """Allocate `out` with torch and run monarch_attn_fwd."""
    import torch

    out = torch.empty_like(q)
    return monarch_attn_fwd(q, k, v, out, m, b, T, stream)


_AUTOGRAD_FN = None


def _autograd_function():
    """torch.autograd.Function whose forward is monarch_attn_fwd (or _varlen)
    and whose backward is monarch_attn_bwd (or _varlen), both on torch's
    current stream."""
    global _AUTOGRAD_FN
    if _AUTOGRAD_FN is None:
        import torch

        class MonarchAttentionFn(torch.autograd.Function):
            @staticmethod
            def forward(ctx, q, k, v, m, b, T, lens):
                q, k, v = q.contiguous(), k.contiguous(), v.contiguous()
                ctx.save_for_backward(q, k, v, lens) if lens is not None else ctx.save_for_backward(q, k, v)
                ctx.shape = (m, b, T)
                out = torch.empty_like(q)
                if lens is None:
                    return monarch_attn_fwd(q, k, v, out, m, b, T)
                return monarch_attn_fwd_varlen(q, k, v, out, lens, m, b, T)

            @staticmethod
            def backward(ctx, dout):
                saved = ctx.saved_tensors
                q, k, v = saved[:3]
                m, b, T = ctx.shape
                dq, dk, dv = (torch.empty_like(q) for _ in range(3))
                if len(saved) == 3:
                    monarch_attn_bwd(q, k, v, dout.contiguous(), dq, dk, dv, m, b, T)
                else:
                    monarch_attn_bwd_varlen(q, k, v, dout.contiguous(), dq, dk, dv, saved[3], m, b, T)
                return dq, dk, dv, None, None, None, None

        _AUTOGRAD_FN = MonarchAttentionFn
    return _AUTOGRAD_FN


def monarch_attention_autograd(q, k, v, m: int, b: int, T: int, lens=None):
    """MonarchAttention as a differentiable torch op: the forward pass and, on
    backward, the gradient with respect to q, k and v.  With lens (int32
    device tensor [B]) the batch is padded per sequence, as in
    monarch_attn_fwd_varlen."""
    return _autograd_function().apply(q, k, v, m, b, T, lens)


def monarch_attn_check(N: int, d: int, m: int, b: int, T: int, dtype: int) -> int:
    return LIB.monarch_attn_check(N, d, m, b, T, dtype)


def fused_applies(d: int, m: int, b: int, dtype: int) -> bool:
    """Whether the one-workgroup-per-head kernel covers this shape."""
    return dtype in (MA_BF16, MA_F16) and d <= 64 and m <= 16 and b <= 16


def grouped_applies(d: int, m: int, b: int, dtype: int) -> bool:
    """Whether the one-workgroup-per-(head, group of classes) kernel (PATH_GROUPED)
    covers this shape (without per-sequence lengths or the objective)."""
    return dtype in (MA_BF16, MA_F16) and d <= 64 and m <= 64 and b <= 32


def monarch_attn_workspace_bytes(B, H, N, d, m, b, T, dtype) -> int:
    return int(LIB.monarch_attn_workspace_bytes(B, H, N, d, m, b, T, dtype))


def monarch_attn_release_workspace() -> None:
    _check(LIB.monarch_attn_release_workspace())


def monarch_attn_set_path(path: int) -> int:
    """Select the execution path (PATH_AUTO, PATH_HALF_STEPS, PATH_FUSED); returns the previous one."""
    prev = LIB.monarch_attn_set_path(path)
    if prev < 0:
        raise MonarchAttnError(MA_EINVAL, monarch_attn_last_error())
    return prev


def monarch_attn_timing_enable(flag: bool) -> None:
    _check(LIB.monarch_attn_timing_enable(1 if flag else 0))


def monarch_attn_timing_read(cap: int = 256):
    """[(kind name, ms), ...] for the launches of the last timed call."""
    ms = (ctypes.c_float * cap)()
    kind = (ctypes.c_int32 * cap)()
    n = LIB.monarch_attn_timing_read(ms, kind, cap)
    if n < 0:
        raise MonarchAttnError(MA_EHIP, monarch_attn_last_error())
    return [(KIND_NAMES.get(kind[i], str(kind[i])), float(ms[i])) for i in range(min(n, cap))]
