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
