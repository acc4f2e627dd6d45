"""Seeded synthetic inputs for the AQLM path.

This module only draws random numbers; it holds none of the method's
arithmetic.  The same bytes feed the GPU library and the CPU oracle.

Distributions stand in for trained checkpoints (paper, App. "Codebook and
codes distribution": learned codes are close to uniform, about 15.91 of 16
bits of entropy, and codebook vectors sit in a ball; scales start at the row
norm in Sec. 3.3, so the codebooks carry the small magnitudes):
  codebooks  N(0, 0.02) rounded to fp16, shape [M, 2^B, g]
  codes      uniform over [0, 2^B), uint8 (B <= 8) or uint16, [d_out, d_in/g, M]
  scales     U[0.5, 1.5] rounded to fp16, [d_out]
  x          N(0, 1) rounded to fp16, [n, d_in]
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Layer:
    codes: np.ndarray      # [d_out, d_in/g, M] uint8 | uint16
    codebooks: np.ndarray  # [M, 2^B, g] float16
    scales: np.ndarray     # [d_out] float16
    x: np.ndarray          # [n, d_in] float16
    M: int
    B: int
    g: int

    @property
    def d_out(self) -> int:
        return self.codes.shape[0]

    @property
    def d_in(self) -> int:
        return self.codes.shape[1] * self.g


def code_dtype(B: int):
    return np.uint8 if B <= 8 else np.uint16


def layer(seed: int, d_out: int, d_in: int, M: int, B: int, g: int = 8, n: int = 1,
          cb_std: float = 0.02) -> Layer:
    """One random AQLM layer plus an input batch, all from ``seed``."""
    if d_in % g:
        raise ValueError("d_in must be a multiple of g")
    rng = np.random.default_rng(seed)
    codebooks = rng.normal(0.0, cb_std, size=(M, 1 << B, g)).astype(np.float16)
    codes = rng.integers(0, 1 << B, size=(d_out, d_in // g, M), dtype=code_dtype(B))
    scales = rng.uniform(0.5, 1.5, size=d_out).astype(np.float16)
    x = rng.standard_normal((n, d_in)).astype(np.float16)
    return Layer(codes, codebooks, scales, x, M, B, g)


# fp16 bit patterns that stress rounding: signed zeros, smallest and largest
# subnormals, smallest normal, values around 1 whose sums land on ties, and
# the largest finite value (sums of it overflow to infinity after scaling).
SPECIAL_F16_BITS = np.array(
    [0x0000, 0x8000, 0x0001, 0x8001, 0x0002, 0x03FF, 0x83FF, 0x0400, 0x8400, 0x0401,
     0x3C00, 0xBC00, 0x3C01, 0x1000, 0x1400, 0x0C00, 0x3800, 0x7BFF, 0xFBFF, 0x7800,
     0x3555, 0xB555, 0x2E66, 0x0200, 0x8200],
    dtype=np.uint16)


def special_layer(seed: int, d_out: int, d_in: int, M: int, B: int, g: int = 8, n: int = 1) -> Layer:
    """A layer whose codebooks and scales mix random finite fp16 bit patterns
    with ``SPECIAL_F16_BITS`` so that dequantized outputs hit fp16 subnormals,
    exact ties, signed zeros and overflow."""
    rng = np.random.default_rng(seed)
    entries = 1 << B
    size = M * entries * g
    raw = rng.integers(0, 1 << 16, size=size, dtype=np.uint32).astype(np.uint16)
    finite = (raw & 0x7C00) != 0x7C00
    raw = np.where(finite, raw, raw & 0x83FF)  # turn inf/NaN patterns into subnormals
    pick = rng.integers(0, SPECIAL_F16_BITS.size, size=size)
    use_special = rng.random(size) < 0.5
    cb_bits = np.where(use_special, SPECIAL_F16_BITS[pick], raw).astype(np.uint16)
    codebooks = cb_bits.reshape(M, entries, g).view(np.float16)
    sc_choices = np.array([0x3C00, 0x3800, 0x3E00, 0x0400, 0x7BFF, 0x0000, 0x8000, 0xBC00,
                           0x3C01, 0x1400, 0x0001, 0x5BFF], dtype=np.uint16)
    sc_bits = np.where(rng.random(d_out) < 0.5, sc_choices[rng.integers(0, sc_choices.size, d_out)],
                       rng.integers(0x0001, 0x7800, d_out).astype(np.uint16)
                       | (rng.integers(0, 2, d_out).astype(np.uint16) << 15))
    scales = sc_bits.astype(np.uint16).view(np.float16)
    codes = rng.integers(0, entries, size=(d_out, d_in // g, M), dtype=code_dtype(B))
    x = rng.standard_normal((n, d_in)).astype(np.float16)
    return Layer(codes, codebooks, scales, x, M, B, g)


def cancelling_layer(seed: int, d_out: int, d_in: int, M: int = 4, g: int = 8, n: int = 1,
                     big: float = 0.5, small: float = 0.004) -> Layer:
    """8-bit codes whose codewords cancel in pairs: codebook 2k holds random
    vectors of size ``big``, codebook 2k + 1 their negations plus a ``small``
    random vector, and the code of codebook 2k + 1 repeats that of 2k.  Every
    weight group is then a small vector built from large codewords, so an
    implementation that rounds partial sums (or per-codebook contributions)
    relative to their own magnitude loses the weight.  M must be even."""
    if M % 2 or d_in % g:
        raise ValueError("M must be even and d_in a multiple of g")
    rng = np.random.default_rng(seed)
    cb = np.empty((M, 256, g), dtype=np.float16)
    codes = np.empty((d_out, d_in // g, M), dtype=np.uint8)
    for k in range(0, M, 2):
        r = rng.normal(0.0, big, size=(256, g)).astype(np.float16)
        cb[k] = r
        cb[k + 1] = (-r.astype(np.float32) + rng.normal(0.0, small, size=(256, g))).astype(np.float16)
        c = rng.integers(0, 256, size=(d_out, d_in // g), dtype=np.uint8)
        codes[:, :, k] = c
        codes[:, :, k + 1] = c
    scales = rng.uniform(0.5, 1.5, size=d_out).astype(np.float16)
    x = rng.standard_normal((n, d_in)).astype(np.float16)
    return Layer(codes, cb, scales, x, M, 8, g)


def device_layer(seed: int, d_out: int, d_in: int, M: int, B: int, g: int = 8, n: int = 1,
                 device="cuda", cb_std: float = 0.02):
    """The same distributions drawn on the GPU with torch's seeded generator
    (for multi-GiB benchmark workloads; the bytes differ from :func:`layer`).
    Returns (codes, codebooks, scales, x) as torch tensors on ``device``;
    codes are uint8 (B <= 8) or int16 holding uint16 bit patterns (B > 8)."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    if B <= 8:
        codes = torch.randint(0, 1 << B, (d_out, d_in // g, M), dtype=torch.uint8, device=device, generator=gen)
    elif B < 16:
        codes = torch.randint(0, 1 << B, (d_out, d_in // g, M), dtype=torch.int16, device=device, generator=gen)
    else:
        codes = torch.randint(-(1 << 15), 1 << 15, (d_out, d_in // g, M), dtype=torch.int16, device=device,
                              generator=gen)
    codebooks = (torch.randn((M, 1 << B, g), device=device, generator=gen) * cb_std).to(torch.float16)
    scales = torch.empty(d_out, device=device).uniform_(0.5, 1.5, generator=gen).to(torch.float16)
    x = torch.randn((n, d_in), device=device, generator=gen).to(torch.float16)
    return codes, codebooks, scales, x


def device_packed_layer(seed: int, d_out: int, d_in: int, M: int, B: int, g: int = 8, n: int = 1,
                        device="cuda", cb_std: float = 0.02):
    """:func:`device_layer` with bit-packed codes: uniformly random 32-bit
    words (every B-bit field of them is a uniform code), int32
    [d_out, ceil(d_in/g * M * B / 32)]."""
    import torch

    _, codebooks, scales, x = device_layer(seed, 8, d_in, M, B, g, n, device, cb_std)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 1)
    words = ((d_in // g) * M * B + 31) // 32
    codes = torch.randint(-(1 << 31), 1 << 31, (d_out, words), dtype=torch.int64, device=device,
                          generator=gen).to(torch.int32)
    scales = torch.empty(d_out, device=device).uniform_(0.5, 1.5, generator=gen).to(torch.float16)
    return codes, codebooks, scales, x
