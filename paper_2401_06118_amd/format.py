"""Shapes and storage accounting of the AQLM format.

Storage model (paper, App. "Estimating model size"): with fp16 codebooks and
scales, one layer costs 16*g*M*2^B bits of codebooks, d_out*(d_in/g)*B*M bits
of codes and 16*d_out bits of scales.  The codes term carries the factor M,
as the App. equation does (the bullet list above it drops it); the paper's
worked example and every bitwidth it prints need it.
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class AqlmShape:
    d_out: int
    d_in: int
    M: int
    B: int
    g: int = 8

    @property
    def groups(self) -> int:
        return self.d_in // self.g

    @property
    def code_bytes_per_group(self) -> int:
        """Bytes the unpacked code tensor spends per group (uint8 or uint16 per code)."""
        return self.M * (1 if self.B <= 8 else 2)

    def storage_bits(self) -> int:
        """Bits of the layer under the paper's storage model (B-bit codes, packed)."""
        return (16 * self.g * self.M * (1 << self.B)
                + self.d_out * self.groups * self.B * self.M
                + 16 * self.d_out)

    def bits_per_param(self) -> float:
        return self.storage_bits() / (self.d_out * self.d_in)

    def codes_bytes(self) -> int:
        """Bytes of the code tensor as the library stores it: one byte per code for
        B <= 8, two for 8 < B <= 16 (unpacked, no padding)."""
        return self.d_out * self.groups * self.code_bytes_per_group

    def paper_codes_bytes(self) -> int:
        """Bytes of the codes at exactly B bits per code (the paper's storage
        count, no padding): d_out * d_in/g * M * B / 8."""
        return self.d_out * self.groups * self.M * self.B // 8

    def paper_gemv_bytes(self, n: int = 1) -> int:
        """:meth:`gemv_bytes` with the codes counted at B bits each."""
        return self.gemv_bytes(n) - self.codes_bytes() + self.paper_codes_bytes()

    def packed_codes_bytes(self) -> int:
        """Bytes of the bit-packed code tensor: B bits per code, each row padded
        to whole 32-bit words."""
        return self.d_out * packed_row_bytes(self.d_in, self.M, self.B, self.g)

    def packed_gemv_bytes(self, n: int = 1) -> int:
        """:meth:`gemv_bytes` with bit-packed codes."""
        return self.gemv_bytes(n) - self.codes_bytes() + self.packed_codes_bytes()

    def codebook_bytes(self) -> int:
        return self.M * (1 << self.B) * self.g * 2

    def gemv_bytes(self, n: int = 1) -> int:
        """Algorithmic HBM bytes of one product with n input rows: codes, codebooks,
        scales, x [n, d_in] and y [n, d_out], each moved once (fp16 activations)."""
        return (self.codes_bytes() + self.codebook_bytes() + 2 * self.d_out
                + 2 * n * self.d_in + 2 * n * self.d_out)

    def dequant_bytes(self) -> int:
        """Algorithmic bytes of dequantization: inputs read once, fp16 W written once."""
        return self.codes_bytes() + self.codebook_bytes() + 2 * self.d_out + 2 * self.d_out * self.d_in

    def flops(self, n: int = 1) -> int:
        return 2 * n * self.d_out * self.d_in


# Linear layers of one transformer block, (d_out, d_in) per projection, in
# the order q, k, v, o, gate, up, down.  Llama-2 architecture shapes.
LLAMA2_BLOCKS = {
    "7b": (32, [(4096, 4096), (4096, 4096), (4096, 4096), (4096, 4096),
                (11008, 4096), (11008, 4096), (4096, 11008)]),
    "13b": (40, [(5120, 5120), (5120, 5120), (5120, 5120), (5120, 5120),
                 (13824, 5120), (13824, 5120), (5120, 13824)]),
    "70b": (80, [(8192, 8192), (1024, 8192), (1024, 8192), (8192, 8192),
                 (28672, 8192), (28672, 8192), (8192, 28672)]),
}


def model_bits_per_param(model: str, M: int, B: int, g: int = 8) -> float:
    """Average bits per parameter over all linear layers of the transformer blocks."""
    n_layers, projs = LLAMA2_BLOCKS[model]
    bits = sum(AqlmShape(o, i, M, B, g).storage_bits() for o, i in projs) * n_layers
    params = sum(o * i for o, i in projs) * n_layers
    return bits / params


def packed_row_bytes(d_in: int, M: int, B: int, g: int = 8) -> int:
    """Bytes of one row of bit-packed codes: G*M codes of B bits, padded to
    whole 32-bit words (the library's packed layout)."""
    return ((d_in // g) * M * B + 31) // 32 * 4


def pack_codes(codes, B: int):
    """Bit-pack codes [d_out, G, M] (values < 2^B): each row's codes in index
    order j*M + m as a little-endian bit string (code q at bits [q*B, (q+1)*B)),
    zero-padded to whole 32-bit words; returns uint8 [d_out, row bytes]."""
    import numpy as np
    c = np.asarray(codes).astype(np.uint64)
    d_out, G, M = c.shape
    n = G * M
    flat = c.reshape(d_out, n)
    pitch = packed_row_bytes(G * 8, M, B)
    bits = ((flat[:, :, None] >> np.arange(B, dtype=np.uint64)[None, None, :]) & 1).astype(np.uint8)
    bits = bits.reshape(d_out, n * B)
    pad = pitch * 8 - n * B
    bits = np.concatenate([bits, np.zeros((d_out, pad), np.uint8)], axis=1)
    return np.packbits(bits.reshape(d_out, pitch, 8), axis=2, bitorder="little").reshape(d_out, pitch)
