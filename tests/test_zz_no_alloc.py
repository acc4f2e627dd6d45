"""aqlm_gemm_noalloc (the product of aqlm_gemm with its workspace in the
library's fixed scratch buffer) through the C ABI, against aqlm_gemm with a
caller workspace: bit-identical outputs on two calls in a row, the second
smaller than the first, plus its error paths."""
import numpy as np
import pytest

import oracle  # noqa: F401  (the oracle check below goes through helpers)
from paper_2401_06118_amd import synth

from helpers import fp16_to_np, to_device

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2401_06118_amd._lib as L
    return L.load()


def noalloc(lib, lay_dev, n, y):
    codes, cb, sc, x = lay_dev
    d_out, G, M = codes.shape
    B = int(cb.shape[1]).bit_length() - 1
    return lib.aqlm_gemm_noalloc(codes.data_ptr(), cb.data_ptr(), sc.data_ptr(), d_out, G * 8, M, B, 8, n,
                                 x.data_ptr(), y.data_ptr(), torch.cuda.current_stream().cuda_stream)


def with_workspace(lay_dev):
    import paper_2401_06118_amd as aq
    codes, cb, sc, x = lay_dev
    return aq.gemm(codes, cb, sc, x)


@pytest.mark.parametrize("first,second", [
    ((11008, 4096, 4, 8, 256), (1000, 2048, 2, 8, 100)),   # 86 MiB of weights, then a small product
    ((4096, 11008, 1, 16, 64), (300, 1024, 4, 8, 64)),    # split along d_in (fp32 partials), then smaller
    ((11000, 576, 2, 8, 1000), (8000, 512, 1, 16, 2000)),  # the dense product's 256-token tiles, fewer weights second
])
def test_noalloc_matches_workspace_product_twice(lib, first, second):
    for k, (d_out, d_in, M, B, n) in enumerate((first, second)):
        print(f"[noalloc] call {k}: {d_out}x{d_in} {M}x{B} n={n}", flush=True)
        lay = synth.layer(31000 + 7 * k + d_out, d_out, d_in, M, B, n=n)
        dev = to_device(lay)
        y = torch.full((n, d_out), float("nan"), dtype=torch.float16, device="cuda")
        assert noalloc(lib, dev, n, y) == 0
        ref = with_workspace(dev)
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy().view(np.uint16), ref.cpu().numpy().view(np.uint16))
        if k == 1:  # the small product against the oracle as well
            from test_gpu_parity import check_products
            check_products(lay, fp16_to_np(y))


def test_noalloc_small_batch_and_refusals(lib):
    """Few rows need no workspace (the call is aqlm_gemm_small_batch); a product
    needing more than the fixed buffer is refused before anything runs."""
    lay = synth.layer(31100, 700, 1024, 2, 8, n=8)
    dev = to_device(lay)
    y = torch.full((8, 700), float("nan"), dtype=torch.float16, device="cuda")
    assert noalloc(lib, dev, 8, y) == 0
    import paper_2401_06118_amd as aq
    ref = aq.gemm_small_batch(*dev)
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy().view(np.uint16), ref.cpu().numpy().view(np.uint16))
    # 12288 x 8192 fp16 weights = 192 MiB > 128 MiB: refused, output untouched
    big = (torch.zeros((12288, 1024, 2), dtype=torch.uint8, device="cuda"), dev[1], 
           torch.ones(12288, dtype=torch.float16, device="cuda"),
           torch.zeros((64, 8192), dtype=torch.float16, device="cuda"))
    yb = torch.full((64, 12288), 3.0, dtype=torch.float16, device="cuda")
    assert noalloc(lib, big, 64, yb) == 7
    torch.cuda.synchronize()
    assert torch.all(yb == 3.0)
