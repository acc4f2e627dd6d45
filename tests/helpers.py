"""Shared test helpers: moving synthetic layers to the GPU and error metrics."""
import numpy as np


def to_device(layer, device="cuda"):
    import torch
    codes = torch.from_numpy(np.ascontiguousarray(layer.codes))
    if layer.codes.dtype == np.uint16:
        codes = torch.from_numpy(np.ascontiguousarray(layer.codes).view(np.int16))
    cb = torch.from_numpy(np.ascontiguousarray(layer.codebooks))
    sc = torch.from_numpy(np.ascontiguousarray(layer.scales))
    x = torch.from_numpy(np.ascontiguousarray(layer.x))
    return codes.to(device), cb.to(device), sc.to(device), x.to(device)


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def fp16_to_np(t):
    return t.detach().cpu().numpy().astype(np.float16)


def assert_bits_equal(got, ref, what=""):
    """uint16 arrays equal bit for bit; on failure report count and a few positions."""
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    bad = np.argwhere(got != ref)
    if bad.size:
        show = ", ".join(f"{tuple(int(v) for v in b)}: {int(got[tuple(b)]):#06x} vs {int(ref[tuple(b)]):#06x}"
                         for b in bad[:6])
        raise AssertionError(f"{what}: {len(bad)} of {ref.size} differ; first: {show}")


def abs_codeword_sums(lay, rows=None):
    """A[i, c] = |s_i| * sum_m |C_m[b_ijm][c mod g]| (fp64) for the listed rows
    (all rows when None): the magnitude of what a kernel adds up before the
    codewords cancel."""
    codes = lay.codes if rows is None else lay.codes[np.asarray(rows)]
    cb = np.abs(lay.codebooks.astype(np.float64))
    acc = cb[0][codes[:, :, 0].astype(np.int64)]
    for m in range(1, codes.shape[2]):
        acc = acc + cb[m][codes[:, :, m].astype(np.int64)]
    sc = np.abs(lay.scales.astype(np.float64))
    if rows is not None:
        sc = sc[np.asarray(rows)]
    return acc.reshape(codes.shape[0], -1) * sc[:, None]


def elementwise_bound(w_bits, x, ref, absw=None):
    """Largest |y_gpu - y_ref| the GPU arithmetic allows for each output.

    With S = sum_c |W[i,c] x[t,c]| over the oracle's fp16 weights W, and
    Sa = sum_c A[i,c] |x[t,c]| over the absolute codeword sums A
    (abs_codeword_sums; Sa = S is used when A is not given):
    - the GPU may skip the fp16 rounding of s_i * (codeword sum): at most
      2^-11 * S (normal range), plus 2^-25 * |x[t,c]| for every W[i,c] in
      the fp16 subnormal range;
    - fp32 accumulation of the codebook contributions over d_in terms in any
      order (and one more rounding inside v_dot2): at most
      2 * d_in * 2^-24 * Sa;
    - the fp16 output: half an ulp, at most 2^-11 * |y| plus 2^-25.
    Codewords that cancel make Sa much larger than S, which is why the
    accumulation term uses it.  Rounding a partial sum of codewords, or a
    codebook's contribution <C_m[b], x_j>, to fp16 is NOT admitted: with
    cancelling codewords its error is relative to a large intermediate, not
    to the weight.
    """
    w = np.abs(w_bits.view(np.float16).astype(np.float64))
    xv = np.asarray(x)
    if xv.dtype == np.uint16:
        xv = xv.view(np.float16)
    xa = np.abs(xv.astype(np.float64).reshape(ref.shape[0], -1))
    d_in = w.shape[1]
    s = xa @ w.T
    sa = s if absw is None else np.maximum(s, xa @ absw.T)
    sub = xa @ (w < 2.0 ** -14).astype(np.float64).T
    return (2.0 ** -11 * np.abs(ref) + 2.1 * 2.0 ** -11 * s + 2 * d_in * 2.0 ** -24 * sa
            + 2.0 ** -25 * sub + 2.0 ** -24)
