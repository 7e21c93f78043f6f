"""Seeded synthetic Q, K, V for the MonarchAttention forward pass.

This module only draws numbers: it holds none of the method's arithmetic, and
both the oracle and the HIP path take their inputs from it.  Every tensor is
[B, H, N, d], drawn as float32 normals from numpy's PCG64 generator seeded by
(seed, crc32(workload/tensor tag)), combined in float32, rounded once to the
run dtype (bf16 and fp16 by round-to-nearest-even), and handed out as float32
arrays holding exactly the rounded values (the oracle widens them to float64).

Recipes (the paper's datasets and pretrained weights are not used; these are
stand-ins with the shapes of its workloads):

* ``iid``   -- Q, K, V iid N(0, 1).
* ``vit``   -- Z, E, V iid N(0, 1); K = Z and Q = 0.7 Z + 0.7 E, which makes
               attention peaky the way a trained ViT's is.
* ``lm``    -- as ``vit`` plus a content vector u ~ N(0, I_d) shared by all
               positions of a (batch, head), then a rotary phase: row p is
               rotated pairwise, (x_2r, x_2r+1) by p * 10000^(-2r/d), so that
               scores decay with |i - j|.
               K_p = rot_p(Z_p + u), Q_p = rot_p(0.7 Z_p + 0.7 E_p + u).
* ``speed`` -- Q, K, V iid N(0, 1), then Q and K both scaled by alpha, where
               alpha is set by bisection so that the mean over 256 sampled
               query rows of the largest softmax(Q K^T / sqrt(d)) weight is
               0.10.
"""
from __future__ import annotations

import dataclasses
import zlib

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "make_qkv",
    "round_to_dtype",
    "bf16_round",
    "DTYPES",
    "random_cotangent",
]

DTYPES = ("f32", "bf16", "f16")


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    m: int
    b: int
    d: int
    T: int
    dtype: str
    recipe: str
    n: int = 0  # sequence length when it is not m * b (post-padded to m * b rows); 0: m * b

    @property
    def N(self) -> int:
        return self.n or self.m * self.b

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "B": self.B,
            "H": self.H,
            "N": self.N,
            "m": self.m,
            "b": self.b,
            "d": self.d,
            "T": self.T,
            "dtype": self.dtype,
            "inputs": self.recipe,
        }


# The workloads: a tiny fp32 parity case, ViT-B/16- and RoBERTa-base-shaped
# attention, the 4K / 16K speed points, and further shapes of the paper's
# conversions.
WORKLOADS = {
    "tiny_f32_n256": Workload("tiny_f32_n256", 1, 1, 16, 16, 64, 1, "f32", "iid"),
    "vit_b16_n196": Workload("vit_b16_n196", 32, 12, 14, 14, 64, 2, "bf16", "vit"),
    # ViT-B/16 with its class token: N = 197, post-padded to 15 blocks of 14
    "vit_b16_n197": Workload("vit_b16_n197", 32, 12, 15, 14, 64, 2, "bf16", "vit", n=197),
    "roberta_n1024": Workload("roberta_n1024", 16, 12, 32, 32, 64, 2, "bf16", "lm"),
    "speed_n4096": Workload("speed_n4096", 1, 16, 64, 64, 64, 1, "bf16", "speed"),
    # the same point at T = 3 (T = 2 is the N = 4096, d = 64 point of the sweep below)
    "speed_n4096_t3": Workload("speed_n4096_t3", 1, 16, 64, 64, 64, 3, "bf16", "speed"),
    "speed_n16384": Workload("speed_n16384", 1, 16, 128, 128, 64, 2, "bf16", "speed"),
    # Shapes of the paper's other conversions, for measurement beside the
    # workloads above (synthetic inputs with the same recipes):
    # DiT-XL/2 at 256 x 256 (16 heads, N = 256, d = 72, b = 16, T = 3), 32 images
    "dit_xl_n256": Workload("dit_xl_n256", 32, 16, 16, 16, 72, 3, "bf16", "vit"),
    # RoBERTa-base on SQuAD at N = 384, T = 1, the b sweep (m = ceil(384 / b))
    "roberta_n384_b24": Workload("roberta_n384_b24", 16, 12, 16, 24, 64, 1, "bf16", "lm"),
    "roberta_n384_b48": Workload("roberta_n384_b48", 16, 12, 8, 48, 64, 1, "bf16", "lm"),
    "roberta_n384_b96": Workload("roberta_n384_b96", 16, 12, 4, 96, 64, 1, "bf16", "lm"),
    "roberta_n384_b128": Workload("roberta_n384_b128", 16, 12, 3, 128, 64, 1, "bf16", "lm"),
    # BART-base encoder (12 heads, d = 64): b = 32 at N = 2048, b = 64 at N = 8192
    "bart_n2048_b32": Workload("bart_n2048_b32", 1, 12, 64, 32, 64, 2, "bf16", "lm"),
    "bart_n8192_b64": Workload("bart_n8192_b64", 1, 12, 128, 64, 64, 2, "bf16", "lm"),
    # 16K tokens with the rotary-decaying scores of the RoBERTa recipe: the
    # approximation-quality point at N = 16384 (the speed points draw iid Q, K,
    # which have no structure for any Monarch matrix to capture)
    "lm_n16384": Workload("lm_n16384", 1, 16, 128, 128, 64, 2, "bf16", "lm"),
    # graph transformer node classification: N = 7600 nodes, b = 128, d = 48
    "gps_n7600": Workload("gps_n7600", 1, 4, 60, 128, 48, 2, "bf16", "vit", n=7600),
}
# The long-sequence sweep: N = 256 .. 16384 in powers of 4 as sqrt(N) x sqrt(N),
# d in {64, 128}, T = 2, the speed recipe (its scale recalibrated for every N).
for _n, _r in ((256, 16), (1024, 32), (4096, 64), (16384, 128)):
    for _d in (64, 128):
        _name = f"sweep_n{_n}_d{_d}"
        WORKLOADS[_name] = Workload(_name, 1, 16, _r, _r, _d, 2, "bf16", "speed")


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16 (nearest, ties to even) via float32; returns float32.

    Finite inputs only (the carry of the rounding add cannot overflow 32 bits).
    """
    f = np.array(x, dtype=np.float32, copy=True, order="C")
    u = f.view(np.uint32)
    bias = (u >> 16) & np.uint32(1)
    bias += np.uint32(0x7FFF)
    u += bias
    u &= np.uint32(0xFFFF0000)
    return f


def round_to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the run dtype; returns float32 holding the rounded values."""
    if dtype == "f32":
        return np.array(x, dtype=np.float32, copy=True, order="C")
    if dtype == "bf16":
        return bf16_round(x)
    if dtype == "f16":
        return np.asarray(x, dtype=np.float32).astype(np.float16).astype(np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def _rng(seed: int, tag: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, zlib.crc32(tag.encode())])))


def _normal(seed: int, tag: str, shape) -> np.ndarray:
    """iid N(0, 1) drawn in float32 (ziggurat)."""
    return _rng(seed, tag).standard_normal(shape, dtype=np.float32)


def _rotary(x: np.ndarray) -> np.ndarray:
    """Rotate pairs (x_2r, x_2r+1) of row p by the angle p * 10000^(-2r/d)."""
    n, d = x.shape[-2], x.shape[-1]
    p = np.arange(n, dtype=np.float64)[:, None]
    r = np.arange(d // 2, dtype=np.float64)[None, :]
    ang = p * np.power(10000.0, -2.0 * r / d)
    c, s = np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)
    x0, x1 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


def _mean_rowmax(sraw: np.ndarray, alpha: float, d: int) -> float:
    z = sraw * (alpha * alpha / np.sqrt(d))
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return float((e.max(axis=1) / e.sum(axis=1)).mean())


def calibrate_alpha(q: np.ndarray, k: np.ndarray, seed: int, target: float = 0.10,
                    rows: int = 256) -> float:
    """Scale making the mean largest softmax weight of sampled rows equal `target`.

    q, k: one head's unscaled [N, d] rows.
    """
    n, d = q.shape
    idx = _rng(seed, "alpha-rows").choice(n, size=min(rows, n), replace=False)
    sraw = q[idx].astype(np.float64) @ k.T.astype(np.float64)
    lo, hi = 0.0, 1.0
    while _mean_rowmax(sraw, hi, d) < target:
        hi *= 2.0
        if hi > 1e3:
            raise RuntimeError("cannot reach the target row-max weight")
    for _ in range(60):
        mid = 0.5 * (lo + hi)
        if _mean_rowmax(sraw, mid, d) < target:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def make_qkv(w: Workload, seed: int = 0):
    """Return (q, k, v, meta): float32 [B, H, N, d] arrays of dtype-rounded values."""
    shape = (w.B, w.H, w.N, w.d)
    tag = f"{w.recipe}/B{w.B}H{w.H}N{w.N}d{w.d}"
    meta = {"seed": seed, "recipe": w.recipe}
    if w.recipe == "iid":
        q = _normal(seed, tag + "/q", shape)
        k = _normal(seed, tag + "/k", shape)
        v = _normal(seed, tag + "/v", shape)
    elif w.recipe in ("vit", "lm"):
        z = _normal(seed, tag + "/z", shape)
        e = _normal(seed, tag + "/e", shape)
        v = _normal(seed, tag + "/v", shape)
        k = z
        q = np.float32(0.7) * z + np.float32(0.7) * e
        if w.recipe == "lm":
            u = _normal(seed, tag + "/u", (w.B, w.H, 1, w.d))
            k = _rotary(k + u)
            q = _rotary(q + u)
    elif w.recipe == "speed":
        q = _normal(seed, tag + "/q", shape)
        k = _normal(seed, tag + "/k", shape)
        v = _normal(seed, tag + "/v", shape)
        alpha = calibrate_alpha(q[0, 0], k[0, 0], seed)
        q *= np.float32(alpha)
        k *= np.float32(alpha)
        meta["alpha"] = alpha
    else:
        raise ValueError(f"unknown recipe {w.recipe!r}")
    q = round_to_dtype(q, w.dtype)
    k = round_to_dtype(k, w.dtype)
    v = round_to_dtype(v, w.dtype)
    return q, k, v, meta


def random_qkv(B, H, N, d, dtype="f32", seed=0, scale=1.0):
    """Plain iid N(0, scale^2) inputs of any shape, for small parity and property cases."""
    tag = f"random/B{B}H{H}N{N}d{d}s{scale}"
    q = round_to_dtype(np.float32(scale) * _normal(seed, tag + "/q", (B, H, N, d)), dtype)
    k = round_to_dtype(np.float32(scale) * _normal(seed, tag + "/k", (B, H, N, d)), dtype)
    v = round_to_dtype(_normal(seed, tag + "/v", (B, H, N, d)), dtype)
    return q, k, v


def sequence_lengths(B: int, N: int, seed: int = 0, low: int = 1) -> np.ndarray:
    """Lengths of a batch of sequences padded to N rows: int32 [B], iid uniform
    on low..N (a stand-in for the length mix of a padded batch)."""
    g = _rng(seed, f"lengths/B{B}N{N}lo{low}")
    return g.integers(low, N + 1, size=B).astype(np.int32)


def random_cotangent(shape, dtype="f32", seed=0, tag="dout"):
    """An iid N(0, 1) tensor of the given shape rounded to the run dtype: the
    incoming gradient dO of a gradient test or benchmark."""
    return round_to_dtype(_normal(seed, f"cotangent/{tag}/{'x'.join(map(str, shape))}", tuple(shape)), dtype)
