"""Seeded synthetic inputs shared by the GPU path's tests/benchmark and the oracle.

This module only draws random numbers; it holds none of the method's
arithmetic.  Every tensor is drawn in float32 from its own numpy PCG64
stream (a SeedSequence keyed by the workload seed and a tensor name) and
rounded to bfloat16 (round to nearest even).  bf16 tensors are returned as
``uint16`` numpy arrays of bit patterns, the form both the oracle and the
C ABI take.

Recipe (stand-ins for the paper's models and text, none of which is used):
hidden states ~ N(0, 1); base weights ~ N(0, w_var); adapter A ~ N(0, 1/d_in)
and B ~ N(0, 0.02) (second argument read as a variance); key outlier
channels are whole rows of W_K (and B_K) multiplied by a factor, so they
flow through the real projection.
"""
from __future__ import annotations

import zlib

import numpy as np
import torch

from .configs import Workload


def stream(seed: int, *names) -> np.random.Generator:
    key = [zlib.crc32(str(n).encode()) for n in names]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal_bf16(seed: int, name, shape, std: float = 1.0) -> np.ndarray:
    x = stream(seed, name).standard_normal(size=shape, dtype=np.float32) * np.float32(std)
    return to_bf16_bits(x)


def key_channel_factors(wl_seed: int, H_kv: int, D: int, outlier) -> np.ndarray:
    """Per-(kv head, channel) multipliers of the key projection rows."""
    g = stream(wl_seed, "outlier")
    f = np.ones((H_kv, D), dtype=np.float32)
    if outlier[0] == "scale":
        _, count, factor = outlier
        for h in range(H_kv):
            idx = g.choice(D, size=count, replace=False)
            f[h, idx] = factor
    elif outlier[0] == "student_t":
        nu = outlier[1]
        f = np.abs(g.standard_t(nu, size=(H_kv, D))).astype(np.float32)
    else:
        raise ValueError(outlier)
    return f


def layer_weights(wl: Workload):
    """(W [d_qkv, d_in], A [3r, d_in], B [d_qkv, r]) as bf16 bits."""
    d_in, r = wl.d_in, wl.rank
    W = stream(wl.seed, "W").standard_normal((wl.d_qkv, d_in), dtype=np.float32)
    W *= np.float32(np.sqrt(wl.w_var))
    fac = key_channel_factors(wl.seed, wl.H_kv, wl.D, wl.outlier).reshape(-1)
    W[wl.d_q:wl.d_q + wl.d_kv] *= fac[:, None]
    A = stream(wl.seed, "A").standard_normal((3 * r, d_in), dtype=np.float32)
    A *= np.float32(np.sqrt(1.0 / d_in))
    Bm = stream(wl.seed, "B").standard_normal((wl.d_qkv, r), dtype=np.float32)
    Bm *= np.float32(np.sqrt(0.02))
    Bm[wl.d_q:wl.d_q + wl.d_kv] *= fac[:, None]
    return to_bf16_bits(W), to_bf16_bits(A), to_bf16_bits(Bm)


def hidden(wl: Workload, name, M: int) -> np.ndarray:
    """Hidden states [M, d_in] ~ N(0, 1) as bf16 bits."""
    return normal_bf16(wl.seed, ("hidden", name), (M, wl.d_in))


def kv_tokens(seed: int, B: int, n: int, H: int, D: int, outlier=("scale", 4, 20.0),
              name="kv"):
    """Stand-alone K, V [B, n, H, D] bf16 bits: V ~ N(0, 1); K ~ N(0, 1) with
    outlier channels (a factor on fixed channels, or i.i.d. Student-t
    entries for the heavy-tailed case)."""
    g = stream(seed, name, "K")
    if outlier is not None and outlier[0] == "student_t":
        K = g.standard_t(outlier[1], size=(B, n, H, D)).astype(np.float32)
    else:
        K = g.standard_normal((B, n, H, D), dtype=np.float32)
        if outlier is not None:
            K *= key_channel_factors(seed, H, D, outlier)[None, None]
    V = stream(seed, name, "V").standard_normal((B, n, H, D), dtype=np.float32)
    return to_bf16_bits(K), to_bf16_bits(V)


def queries(seed: int, B: int, H_q: int, D: int, name="q") -> np.ndarray:
    return normal_bf16(seed, ("q", name), (B, H_q, D))


def normal_bf16_device(seed: int, name, shape, device="cuda", std: float = 1.0):
    """Large ~N(0, std^2) bf16 tensors drawn directly on the device (torch's
    Philox generator, seeded from the same SeedSequence keys); used for
    benchmark inputs that the oracle never consumes."""
    key = int(stream(seed, "device", name).integers(0, 2 ** 62))
    g = torch.Generator(device=device)
    g.manual_seed(key)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x *= std
    return x.to(torch.bfloat16)
