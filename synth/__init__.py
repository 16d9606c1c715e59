"""Seeded synthetic inputs for the Fairy2i widely-linear layer.

This module only draws random numbers: real weight matrices with the shapes
and value distribution of LLaMA-2-7B's linear layers, complex activations
~ N(0, 1), and their rounding to bf16.  It holds none of the method's
arithmetic (no widely-linear transform, no quantisation, no products), so the
CPU oracle and the GPU path can both be fed from it without sharing any of the
computation they are checked on.

Conventions
-----------
* A real layer is ``A`` of shape (2N, 2K), float32, row = output, column =
  input (the paper's R in its real-layer equation, Sec. 3.1).
* A complex activation batch is ``x`` of shape (B, K), complex64.  It is drawn
  as a real vector x~ in R^{2K} per token and paired as
  x = x~[:K] + i x~[K:] (the stacked real/imaginary halves of Sec. 3.1).
* bf16 activations are produced by round-to-nearest-even of the float32
  draws; ``bf16_round`` returns the rounded values as float32 (exactly
  representable), ``bf16_bits`` the raw 16-bit patterns.
"""
from __future__ import annotations

import numpy as np

# LLaMA-2-7B linear layer shapes (real out x in) per decoder layer.
LLAMA2_7B_PROJ = {
    "q": (4096, 4096),
    "k": (4096, 4096),
    "v": (4096, 4096),
    "o": (4096, 4096),
    "gate": (11008, 4096),
    "up": (11008, 4096),
    "down": (4096, 11008),
}
PROJ_ORDER = ("q", "k", "v", "o", "gate", "up", "down")
N_LAYERS = 32


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(list(key)))


def small_layer() -> tuple[np.ndarray, np.ndarray]:
    """The 256x256 single-layer case.

    A has i.i.d. N(0, 1/256) float32 entries drawn from ``default_rng(0)``;
    the same stream then gives one real activation x~ in R^256 ~ N(0,1),
    paired into x in C^128.  Returns (A [256,256] float32, x [1,128] complex64).
    """
    rng = np.random.default_rng(0)
    A = (rng.standard_normal((256, 256)) / 16.0).astype(np.float32)
    xt = rng.standard_normal(256).astype(np.float32)
    x = (xt[:128].astype(np.complex64) + 1j * xt[128:].astype(np.complex64))
    return A, x.reshape(1, 128).astype(np.complex64)


def llama_weight(rows: int, cols: int, key: tuple[int, ...],
                 outlier_frac: float = 0.01, outlier_mult: float = 10.0,
                 std: float = 0.02) -> np.ndarray:
    """LLaMA-like synthetic real weight, float32 [rows, cols].

    Entries are Student-t with 4 degrees of freedom scaled to standard
    deviation ``std`` (t_4 has variance 2, so the scale is std/sqrt(2)); then
    round(outlier_frac * cols) distinct input channels (columns), chosen by the
    same seeded stream, are multiplied by ``outlier_mult``.
    """
    rng = _rng(*key)
    A = rng.standard_t(4, size=(rows, cols)) * (std / np.sqrt(2.0))
    n_out = int(round(outlier_frac * cols))
    if n_out:
        idx = rng.choice(cols, size=n_out, replace=False)
        A[:, idx] *= outlier_mult
    return A.astype(np.float32)


def activations(batch: int, k: int, key: tuple[int, ...]) -> np.ndarray:
    """B tokens of complex activations, complex64 [batch, k].

    Each token is a real N(0,1) float32 vector of length 2k paired as
    x = x~[:k] + i x~[k:].
    """
    rng = _rng(*key)
    xt = rng.standard_normal((batch, 2 * k)).astype(np.float32)
    return (xt[:, :k].astype(np.complex64) + 1j * xt[:, k:].astype(np.complex64)).astype(np.complex64)


def bf16_bits(v: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); uint16 patterns."""
    u = np.ascontiguousarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact float32 values of bf16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_round(v: np.ndarray) -> np.ndarray:
    """float32 array holding the bf16-rounded values of ``v``."""
    return bf16_to_f32(bf16_bits(v))


def bf16_round_complex(x: np.ndarray) -> np.ndarray:
    """Round the real and imaginary parts of a complex64 array to bf16."""
    re = bf16_round(x.real.astype(np.float32))
    im = bf16_round(x.imag.astype(np.float32))
    return (re.astype(np.complex64) + 1j * im.astype(np.complex64)).astype(np.complex64)


def layer_key(config: int, layer: int, proj: str) -> tuple[int, int, int]:
    return (config, layer, PROJ_ORDER.index(proj))


def torch_llama_weight(rows: int, cols: int, seed: int, device,
                       outlier_frac: float = 0.01, outlier_mult: float = 10.0,
                       std: float = 0.02):
    """Same distribution as ``llama_weight`` drawn with torch's generator on
    ``device`` (used for the 224-layer stack, where drawing 6.5e9 samples on
    the host would take minutes).  A different stream from ``llama_weight``."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    # Student-t(4) = Z / sqrt(V/4) with V ~ chi^2_4 = sum of 4 squared normals.
    z = torch.randn(rows, cols, generator=g, device=device, dtype=torch.float32)
    v = torch.zeros(rows, cols, device=device, dtype=torch.float32)
    for _ in range(4):
        e = torch.randn(rows, cols, generator=g, device=device, dtype=torch.float32)
        v.addcmul_(e, e)
    A = z * torch.rsqrt(v * 0.25) * (std / 2.0 ** 0.5)
    n_out = int(round(outlier_frac * cols))
    if n_out:
        idx = torch.randperm(cols, generator=g, device=device)[:n_out]
        A[:, idx] *= outlier_mult
    return A.contiguous()
