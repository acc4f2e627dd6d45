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


def elementwise_bound(w_bits, x, ref):
    """Largest |y_gpu - y_ref| the GPU arithmetic allows for each output.

    With S = sum_c |W[i,c] x[t,c]| over the oracle's fp16 weights W:
    - the GPU may skip the fp16 rounding of s_i * (codeword sum), or round
      fp16 partial products: at most 2^-11 * S each (normal range), plus
      2^-25 * |x[t,c]| for every W[i,c] in the fp16 subnormal range;
    - fp32 accumulation over d_in terms in any order (and one more rounding
      inside v_dot2): at most 2 * d_in * 2^-24 * S;
    - the fp16 output: half an ulp, at most 2^-11 * |y| plus 2^-25.
    """
    w = np.abs(w_bits.view(np.float16).astype(np.float64))
    xv = np.asarray(x)
    if xv.dtype == np.uint16:
        xv = xv.view(np.float16)
    xa = np.abs(xv.astype(np.float64).reshape(ref.shape[0], -1))
    d_in = w.shape[1]
    s = xa @ w.T
    sub = xa @ (w < 2.0 ** -14).astype(np.float64).T
    return 2.0 ** -11 * np.abs(ref) + (2.1 * 2.0 ** -11 + 2 * d_in * 2.0 ** -24) * s + 2.0 ** -25 * sub + 2.0 ** -24
