"""CPU checks of the elementwise error bound the GPU product tests apply
(helpers.elementwise_bound): it admits every result that GPU-style
arithmetic can produce, and it rejects results with one plausible kernel
mistake planted in them."""
import numpy as np
import pytest

import oracle
from helpers import abs_codeword_sums, elementwise_bound
from paper_2401_06118_amd import synth


def _f32(a):
    a = np.asarray(a)
    return (a.view(np.float16) if a.dtype == np.uint16 else a).astype(np.float32)


def gpu_like(lay, *, drop=None, scale_shift=0, fp16_partials=False, fp16_table=False):
    """Y = fp16(s_i * sum_c u[i,c] x[t,c]) with u the fp32 codeword sums, never
    rounded to fp16, and fp32 accumulation in 64 blocks along d_in (an order
    unlike the oracle's).  drop = (row, first input, count) leaves those inputs
    of one row out; scale_shift = k uses row i + k's scale for row i.
    fp16_partials: the codewords are added with fp16 adds (each partial sum
    rounded to fp16).  fp16_table: each codebook's contribution
    <C_m[b_ijm], x_j> is rounded to fp16 (a partial-product table) and those
    are accumulated in fp32."""
    d_out, G, M = lay.codes.shape
    cb = _f32(lay.codebooks)
    codes = lay.codes.astype(np.int64)
    x = _f32(lay.x)
    n = x.shape[0]
    s = np.roll(_f32(lay.scales), -scale_shift)
    if fp16_table:
        xg = x.reshape(n, G, 8)
        acc = np.zeros((n, d_out), np.float32)
        for m in range(M):
            cw = cb[m][codes[:, :, m]]                                       # [d_out, G, 8]
            t = np.einsum("igk,tgk->tig", cw.astype(np.float64), xg.astype(np.float64))
            t = t.astype(np.float32).astype(np.float16).astype(np.float32)   # fp16 table entries
            acc = (acc + t.reshape(n, d_out, 64, -1).sum(axis=3, dtype=np.float32).sum(axis=2, dtype=np.float32))
        return (acc * s[None, :]).astype(np.float32).astype(np.float16).astype(np.float64)
    u = cb[0][codes[:, :, 0]]
    for m in range(1, M):
        if fp16_partials:
            u = (u.astype(np.float16) + cb[m][codes[:, :, m]].astype(np.float16)).astype(np.float32)
        else:
            u = (u + cb[m][codes[:, :, m]]).astype(np.float32)
    u = u.reshape(d_out, G * 8)
    if drop is not None:
        row, c0, cnt = drop
        u = u.copy()
        u[row, c0:c0 + cnt] = 0.0
    prod = (u[None, :, :] * x[:, None, :]).astype(np.float32)
    acc = prod.reshape(n, d_out, 64, -1).sum(axis=3, dtype=np.float32).sum(axis=2, dtype=np.float32)
    return (acc * s[None, :]).astype(np.float32).astype(np.float16).astype(np.float64)


def _violations(lay, y):
    w = oracle.dequantize(lay.codes, lay.codebooks, lay.scales)
    ref = oracle.matmul_f16(w, lay.x)
    return np.abs(y - ref) > elementwise_bound(w, lay.x, ref, abs_codeword_sums(lay))


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


@pytest.mark.parametrize("M", [2, 4])
def test_bound_admits_fp32_sums_of_cancelling_codewords(M):
    lay = synth.cancelling_layer(61 + M, 96, 2048, M, n=2)
    assert not _violations(lay, gpu_like(lay)).any()


def _rel_l2(lay, y):
    ref = oracle.matmul_f16(oracle.dequantize(lay.codes, lay.codebooks, lay.scales), lay.x)
    return float(np.linalg.norm(y - ref) / np.linalg.norm(ref))


@pytest.mark.parametrize("mode", ["fp16_partials", "fp16_table"])
def test_fp16_intermediates_fail_acceptance_on_cancelling_codewords(mode):
    """Codebooks that cancel in pairs: rounding the codeword partial sums, or
    each codebook's contribution <C_m[b], x_j>, to fp16 loses much of the
    small weight, and the result misses the 2e-3 relative-L2 acceptance
    while fp32 intermediates meet it by a wide margin.  This is why the
    kernels add codewords, and partial-product table entries, in fp32."""
    lay = synth.cancelling_layer(71, 96, 2048, 4, n=2)
    assert _rel_l2(lay, gpu_like(lay)) < 1e-3
    assert _rel_l2(lay, gpu_like(lay, **{mode: True})) > 5e-3


def test_cancelling_layer_makes_small_weights():
    lay = synth.cancelling_layer(72, 32, 256, 4)
    w = np.abs(_f32(oracle.dequantize(lay.codes, lay.codebooks, lay.scales)))
    assert np.median(w) < 0.02 * np.median(np.abs(_f32(lay.codebooks)))
