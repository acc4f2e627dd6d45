"""CPU checks of the elementwise error bound the GPU product tests apply
(helpers.elementwise_bound): it admits every result that GPU-style
arithmetic can produce, and it rejects results with one plausible kernel
mistake planted in them."""
import numpy as np
import pytest

import oracle
from helpers import elementwise_bound
from paper_2401_06118_amd import synth


def _f32(a):
    a = np.asarray(a)
    return (a.view(np.float16) if a.dtype == np.uint16 else a).astype(np.float32)


def gpu_like(lay, *, drop=None, scale_shift=0):
    """Y = fp16(s_i * sum_c u[i,c] x[t,c]) with u the fp32 codeword sums, never
    rounded to fp16, and fp32 accumulation in 64 blocks along d_in (an order
    unlike the oracle's).  drop = (row, first input, count) leaves those inputs
    of one row out; scale_shift = k uses row i + k's scale for row i."""
    d_out, G, M = lay.codes.shape
    cb = _f32(lay.codebooks)
    codes = lay.codes.astype(np.int64)
    u = cb[0][codes[:, :, 0]]
    for m in range(1, M):
        u = (u + cb[m][codes[:, :, m]]).astype(np.float32)
    u = u.reshape(d_out, G * 8)
    if drop is not None:
        row, c0, cnt = drop
        u = u.copy()
        u[row, c0:c0 + cnt] = 0.0
    x = _f32(lay.x)
    n = x.shape[0]
    prod = (u[None, :, :] * x[:, None, :]).astype(np.float32)
    acc = prod.reshape(n, d_out, 64, -1).sum(axis=3, dtype=np.float32).sum(axis=2, dtype=np.float32)
    s = np.roll(_f32(lay.scales), -scale_shift)
    return (acc * s[None, :]).astype(np.float32).astype(np.float16).astype(np.float64)


def _violations(lay, y):
    w = oracle.dequantize(lay.codes, lay.codebooks, lay.scales)
    ref = oracle.matmul_f16(w, lay.x)
    return np.abs(y - ref) > elementwise_bound(w, lay.x, ref)


@pytest.mark.parametrize("d_out,d_in,M,B,n", [(64, 4096, 2, 8, 1), (32, 11008, 1, 16, 2), (48, 2048, 4, 8, 3),
                                              (16, 28672, 2, 8, 1)])
def test_bound_admits_gpu_style_arithmetic(d_out, d_in, M, B, n):
    lay = synth.layer(31 + d_in, d_out, d_in, M, B, n=n)
    assert not _violations(lay, gpu_like(lay)).any()


def test_bound_rejects_one_dropped_k_slice():
    """One 64-byte K-slice (32 groups, 256 inputs) of one row left out: the
    slice of row 100 whose terms add up to the most."""
    lay = synth.layer(57, 256, 4096, 2, 8)
    w = _f32(oracle.dequantize(lay.codes, lay.codebooks, lay.scales))
    contrib = (w[100] * _f32(lay.x)[0]).reshape(-1, 256).sum(axis=1)
    k = int(np.argmax(np.abs(contrib)))
    bad = _violations(lay, gpu_like(lay, drop=(100, 256 * k, 256)))
    assert bad[0, 100] and bad.sum() == 1


def test_bound_rejects_scales_of_the_next_row():
    lay = synth.layer(58, 256, 4096, 2, 8)
    assert _violations(lay, gpu_like(lay, scale_shift=1)).sum() > 128
