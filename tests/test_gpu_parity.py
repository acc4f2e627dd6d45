"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Dequantization must match the oracle bit for bit (uint16 patterns, signed
zeros included).  Products must be within relative L2 error 2e-3 of the
oracle's fp64 result, per activation row and over the whole output.
"""
import numpy as np
import pytest

import oracle
from paper_2401_06118_amd import synth

from helpers import abs_codeword_sums, assert_bits_equal, elementwise_bound, fp16_to_np, rel_l2, to_device

pytestmark = pytest.mark.gpu
TOL = 2e-3

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2401_06118_amd._lib as L
    L.load()  # raises if the HIP library is missing: no fallback


def aq():
    import paper_2401_06118_amd as m
    return m


def dequant_gpu(lay):
    codes, cb, sc, _ = to_device(lay)
    w = aq().dequantize(codes, cb, sc)
    torch.cuda.synchronize()
    return w.cpu().numpy().view(np.uint16)


def check_products(lay, y_gpu, rows=None):
    """y_gpu: [n, d_out] fp16 numpy.  rows: optional sampled row indices.

    Passes when every token row and the whole output are within relative L2
    error TOL of the oracle, and every element is within the bound its
    arithmetic allows (elementwise_bound)."""
    if rows is None:
        w = oracle.dequantize(lay.codes, lay.codebooks, lay.scales, lay.g)
        got = y_gpu
    else:
        w = oracle.dequantize_rows(lay.codes, lay.codebooks, lay.scales, rows, lay.g)
        got = y_gpu[:, rows]
    ref = oracle.matmul_f16(w, lay.x)
    assert np.all(np.isfinite(got.astype(np.float64)))
    for t in range(ref.shape[0]):
        assert rel_l2(got[t], ref[t]) <= TOL, (t, rel_l2(got[t], ref[t]))
    assert rel_l2(got, ref) <= TOL
    err = np.abs(got.astype(np.float64) - ref)
    bound = elementwise_bound(w, lay.x, ref, abs_codeword_sums(lay, rows))
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert np.all(err <= bound), ("elementwise", worst, err[worst], bound[worst])


# ------------------------------------------------------------------ dequantize

DEQ_CASES = [
    # (d_out, d_in, M, B)
    (4096, 4096, 2, 8),     # 2x8 layer
    (4096, 4096, 1, 16),    # 1x16 layer
    (1000, 4104, 4, 8),
    (3, 24, 1, 8), (1, 8, 3, 8), (17, 40, 5, 8), (33, 136, 6, 8), (64, 64, 7, 8), (100, 512, 8, 8),
    (1, 8, 1, 16), (1000, 24, 1, 16),
]


@pytest.mark.parametrize("d_out,d_in,M,B", DEQ_CASES)
def test_dequantize_bit_exact(d_out, d_in, M, B):
    print(f"[dequant] d_out={d_out} d_in={d_in} M={M} B={B}", flush=True)
    lay = synth.layer(1000 + d_out + M, d_out, d_in, M, B)
    assert_bits_equal(dequant_gpu(lay), oracle.dequantize(lay.codes, lay.codebooks, lay.scales), "dequantize")


@pytest.mark.parametrize("M,B", [(1, 8), (2, 8), (3, 8), (4, 8), (8, 8), (1, 16), (2, 12)])
def test_dequantize_special_values_bit_exact(M, B):
    """Codebooks and scales mixing random finite fp16 patterns with signed
    zeros, subnormals, ties and values whose scaled sums overflow."""
    print(f"[dequant-special] M={M} B={B}", flush=True)
    lay = synth.special_layer(77 + M, 257, 136, M, B)
    got = dequant_gpu(lay)
    ref = oracle.dequantize(lay.codes, lay.codebooks, lay.scales)
    assert_bits_equal(got, ref, "dequantize special")
    # the fixture does reach the interesting encodings
    assert np.any(ref == 0x8000) and np.any((ref & 0x7C00) == 0) and np.any((ref & 0x7FFF) == 0x7C00)


def test_dequantize_large_layer_sampled_rows():
    """11008 x 4096 with four codebooks (the prefill layer), rows sampled."""
    print("[dequant] 11008x4096 4x8", flush=True)
    lay = synth.layer(4242, 11008, 4096, 4, 8)
    got = dequant_gpu(lay)
    rows = np.array([0, 1, 4095, 5503, 11006, 11007] + list(range(100, 11008, 997)))
    ref = oracle.dequantize_rows(lay.codes, lay.codebooks, lay.scales, rows)
    assert_bits_equal(got[rows], ref, "dequantize rows")


def test_dequantize_is_deterministic():
    lay = synth.layer(5, 512, 1024, 2, 8)
    a = dequant_gpu(lay)
    b = dequant_gpu(lay)
    assert np.array_equal(a, b)


# ------------------------------------------------------------------------ GEMV

GEMV_CASES = [
    (4096, 4096, 2, 8),
    (4096, 4096, 1, 16),
    (11008, 4096, 1, 16),
    (4096, 11008, 1, 16),
    (4096, 11008, 2, 8),
    (11008, 4096, 4, 8),
    (1, 8, 2, 8), (3, 24, 1, 8), (1000, 4104, 2, 8), (1000, 4104, 1, 16), (5, 8192, 1, 16),
    (64, 512, 3, 8), (70, 1024, 5, 8), (130, 1040, 6, 8), (31, 2048, 7, 8), (257, 4096, 8, 8), (129, 4096, 1, 8),
]


@pytest.mark.parametrize("d_out,d_in,M,B", GEMV_CASES)
def test_gemv_matches_oracle(d_out, d_in, M, B):
    print(f"[gemv] d_out={d_out} d_in={d_in} M={M} B={B}", flush=True)
    lay = synth.layer(2000 + d_out + d_in + M, d_out, d_in, M, B)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y)[None, :])


@pytest.mark.parametrize("shapes", [
    [(11001, 4096)],            # ragged rows, one K-slice per wave, 3 row blocks per workgroup
    [(8192, 6144)],             # two K-slices per wave
    [(5000, 12288)],            # three K-slices per wave (the largest d_in staged next to a chunk)
    [(5000, 12352)],            # one more K-slice: falls back to the L2 gathers
    [(11008, 4096)] * 2,        # gate/up: 6 row blocks per workgroup
    [(4096, 4096), (1024, 4096), (12000, 4096)],  # grouped, above the size threshold together
    [(11008, 4096), (4096, 11008)],                # grouped with different d_in: the first problem's
                                                   # waves carry two empty K-slices (x zero there)
])
def test_gemv_1x16_codebook_chunks(shapes):
    """1x16 launches large enough for the kernel that stages the codebook in
    LDS chunk by chunk (eight passes, zero codeword outside the chunk)."""
    print(f"[gemv-1x16-chunks] {shapes}", flush=True)
    if len(shapes) == 1:
        d_out, d_in = shapes[0]
        lay = synth.layer(9100 + d_out + d_in, d_out, d_in, 1, 16)
        codes, cb, sc, x = to_device(lay)
        y = aq().gemv(codes, cb, sc, x[0])
        torch.cuda.synchronize()
        check_products(lay, fp16_to_np(y)[None, :])
    else:
        _grouped_case(shapes, 1, 16, 9200)


@pytest.mark.parametrize("shapes", [[(300, 20480)], [(1000, 16384)], [(77, 28672)], [(512, 16384), (96, 20480)]])
def test_gemv_eight_codebook_copies(shapes):
    """2x8 layers wide enough that x leaves room for only 8 codebook copies:
    the interleaved copy layout where lanes 8-15 gather the other codebook."""
    print(f"[gemv-8copies] {shapes}", flush=True)
    if len(shapes) == 1:
        lay = synth.layer(3100 + shapes[0][1], shapes[0][0], shapes[0][1], 2, 8)
        codes, cb, sc, x = to_device(lay)
        check_products(lay, fp16_to_np(aq().gemv(codes, cb, sc, x[0]))[None, :])
    else:
        _grouped_case(shapes, 2, 8, 3200)


def test_gemv_70b_shapes_sampled_rows():
    """Llama-2-70B-shaped 2x8 layers: gate/up 28672 x 8192, down 8192 x 28672,
    k/v 1024 x 8192; outputs checked on sampled rows."""
    for d_out, d_in in [(28672, 8192), (8192, 28672), (1024, 8192)]:
        print(f"[gemv-70b] {d_out}x{d_in}", flush=True)
        lay = synth.layer(3000 + d_out, d_out, d_in, 2, 8)
        codes, cb, sc, x = to_device(lay)
        y = fp16_to_np(aq().gemv(codes, cb, sc, x[0]))[None, :]
        rows = np.unique(np.concatenate([[0, d_out - 1], np.random.default_rng(1).integers(0, d_out, 96)]))
        check_products(lay, y, rows)


@pytest.mark.parametrize("M,B", [(2, 8), (1, 16)])
def test_gemv_deterministic(M, B):
    """100 repeated products give bit-identical outputs."""
    lay = synth.layer(9, 4096, 4096, M, B)
    codes, cb, sc, x = to_device(lay)
    ys = torch.stack([aq().gemv(codes, cb, sc, x[0]) for _ in range(100)])
    ys = ys.cpu().numpy().view(np.uint16)
    assert (ys == ys[0]).all()


@pytest.mark.parametrize("n", [1, 4, 16, 40, 256])
@pytest.mark.parametrize("M", [2, 4])
def test_cancelling_codewords_all_products(n, M):
    """Codebooks that cancel in pairs (small weights built from large
    codewords) through the matrix-vector, small-batch, chunked, fused-prefill
    and workspace products: the codeword sums must not lose the weight."""
    print(f"[cancelling] n={n} M={M}", flush=True)
    lay = synth.cancelling_layer(9000 + 10 * n + M, 1000, 2048, M, n=n)
    codes, cb, sc, x = to_device(lay)
    y1 = aq().gemm_small_batch(codes, cb, sc, x)
    y2 = aq().gemm(codes, cb, sc, x)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y1))
    check_products(lay, fp16_to_np(y2))
    assert_bits_equal(dequant_gpu(lay), oracle.dequantize(lay.codes, lay.codebooks, lay.scales), "dequantize")


def test_gemv_zero_scales_give_zero():
    lay = synth.layer(10, 512, 1024, 2, 8)
    lay.scales[:] = 0
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0]).cpu().numpy()
    assert np.all(y == 0)


def test_gemv_identity_codebook_is_plain_fp16_matvec():
    """M = 1, B = 16 with the 65536 fp16 groups of a matrix W as the codebook:
    the product must agree with the fp64 product of W itself."""
    rng = np.random.default_rng(11)
    w = rng.standard_normal((256, 2048)).astype(np.float16)
    lay = synth.layer(0, 256, 2048, 1, 16)
    lay.codebooks = w.reshape(1, 65536, 8)
    lay.codes = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(256, 256, 1)
    lay.scales = np.ones(256, np.float16)
    codes, cb, sc, x = to_device(lay)
    y = fp16_to_np(aq().gemv(codes, cb, sc, x[0]))
    ref = w.astype(np.float64) @ lay.x[0].astype(np.float64)
    assert rel_l2(y, ref) <= TOL


# ------------------------------------------------------------ small batch / MFMA

@pytest.mark.parametrize("n", list(range(1, 21)) + [31, 64, 255, 256, 257])
@pytest.mark.parametrize("M,B", [(2, 8), (1, 16), (4, 8)])
def test_gemm_small_batch_matches_oracle(n, M, B):
    print(f"[gemm] n={n} M={M} B={B}", flush=True)
    lay = synth.layer(5000 + n * 10 + M, 1000, 1040, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemm_small_batch(codes, cb, sc, x)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y))


@pytest.mark.parametrize("M", [1, 3, 5, 6, 7, 8])
def test_gemm_small_batch_other_codebook_counts(M):
    lay = synth.layer(6000 + M, 200, 520, M, 8, n=5)
    codes, cb, sc, x = to_device(lay)
    check_products(lay, fp16_to_np(aq().gemm_small_batch(codes, cb, sc, x)))


@pytest.mark.parametrize("n", [16, 2048])
@pytest.mark.parametrize("M,B", [(1, 16), (4, 8)])
def test_prefill_layer_sampled_rows(n, M, B):
    """11008 x 4096 with n in {16, 2048} activation rows, sampled output rows."""
    print(f"[prefill] n={n} M={M} B={B}", flush=True)
    lay = synth.layer(7000 + n + M, 11008, 4096, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    y = fp16_to_np(aq().gemm_small_batch(codes, cb, sc, x))
    rows = np.unique(np.concatenate([[0, 11007], np.random.default_rng(2).integers(0, 11008, 40)]))
    check_products(lay, y, rows)


@pytest.mark.parametrize("d_out,d_in,M,n", [
    (1000, 4096, 2, 2), (1000, 4096, 2, 16), (1000, 4096, 4, 5), (1000, 4096, 4, 16),
    (300, 11008, 4, 3), (300, 11008, 4, 16), (300, 11008, 2, 16), (4100, 2048, 4, 7),
    (17, 264, 4, 9), (16, 4096, 2, 4),
])
def test_gemm_small_batch_shapes(d_out, d_in, M, n):
    """2..16 tokens over several K-slice rounds, ragged rows, aligned and
    unaligned code pitches, and the LDS budgets of n = 16."""
    print(f"[gemm-nb] {d_out}x{d_in} M={M} n={n}", flush=True)
    lay = synth.layer(5500 + d_out + d_in + M + n, d_out, d_in, M, 8, n=n)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemm_small_batch(codes, cb, sc, x)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y))


@pytest.mark.parametrize("d_out,d_in,M,B,n", [
    (300, 1040, 2, 8, 17), (300, 1040, 4, 8, 300), (129, 520, 1, 8, 40), (1000, 4096, 2, 8, 256),
    (1000, 4096, 4, 8, 513), (260, 4104, 1, 16, 100), (128, 64, 4, 8, 257), (4096, 512, 2, 8, 1024),
    (7, 2056, 1, 16, 33),
])
def test_prefill_shapes(d_out, d_in, M, B, n):
    """Many tokens: ragged row and token tiles, K not a multiple of the
    64-input step, aligned and unaligned code pitches, every format."""
    print(f"[prefill-shapes] {d_out}x{d_in} M={M} B={B} n={n}", flush=True)
    lay = synth.layer(5800 + d_out + d_in + M + B + n, d_out, d_in, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemm_small_batch(codes, cb, sc, x)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y))


def test_prefill_deterministic():
    lay = synth.layer(15, 700, 2048, 4, 8, n=300)
    codes, cb, sc, x = to_device(lay)
    ys = torch.stack([aq().gemm_small_batch(codes, cb, sc, x) for _ in range(100)]).cpu().numpy().view(np.uint16)
    assert (ys == ys[0]).all()


@pytest.mark.parametrize("d_out,d_in,M,B", [(24, 40960, 2, 8), (40, 40968, 4, 8), (17, 65544, 1, 16), (8, 131072, 1, 8)])
def test_gemv_wide_layers(d_out, d_in, M, B):
    """d_in beyond what the matrix-core kernel stages in LDS: the vector-ALU
    kernel takes over (also through the grouped entry point)."""
    print(f"[gemv-wide] {d_out}x{d_in} M={M} B={B}", flush=True)
    lay = synth.layer(5900 + d_in + M, d_out, d_in, M, B)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    y2 = torch.empty_like(y)
    aq().gemv_grouped([(codes, cb, sc, x[0], y2)])
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y)[None])
    check_products(lay, fp16_to_np(y2)[None])


# ------------------------------------------------- workspace product (aqlm_gemm)

@pytest.mark.parametrize("d_out,d_in,M,B,n", [
    (1000, 4096, 2, 8, 64), (300, 1024, 4, 8, 300), (129, 512, 1, 16, 257), (4096, 4160, 1, 16, 100),
    (130, 1024, 3, 8, 65), (257, 512, 8, 8, 513), (1, 64, 2, 8, 64), (64, 64, 1, 8, 1000),
    (4096, 11008, 4, 8, 64), (200, 2048, 2, 8, 130),
])
def test_gemm_workspace_matches_oracle(d_out, d_in, M, B, n):
    """Two-pass path: ragged token and row tiles, every format (the weights
    are rebuilt by the dequantization kernel, so M = 3 and 8 work too), and
    products split along K (few tiles: 2 to 8 splits)."""
    print(f"[gemm-ws] {d_out}x{d_in} M={M} B={B} n={n}", flush=True)
    lay = synth.layer(8200 + d_out + d_in + M + B + n, d_out, d_in, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    need = aq().gemm_workspace_bytes(codes, cb, sc, n)
    assert need >= d_out * d_in * 2  # plus fp32 partial sums when the product is split along K
    ws = torch.full((need,), 0xAB, dtype=torch.uint8, device="cuda")
    y = aq().gemm(codes, cb, sc, x, workspace=ws)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y))
    # the workspace starts with the dequantized weights, bit for bit
    w = ws[: d_out * d_in * 2].view(torch.float16).view(d_out, d_in).cpu().numpy().view(np.uint16)
    assert_bits_equal(w, oracle.dequantize(lay.codes, lay.codebooks, lay.scales))


@pytest.mark.parametrize("n", [2048])
@pytest.mark.parametrize("M,B", [(1, 16), (4, 8)])
def test_gemm_workspace_prefill_layer_sampled_rows(n, M, B):
    """11008 x 4096 with 2048 activation rows (the prefill workload), sampled
    output rows against the oracle."""
    print(f"[gemm-ws prefill] n={n} M={M} B={B}", flush=True)
    lay = synth.layer(7000 + n + M, 11008, 4096, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    y = fp16_to_np(aq().gemm(codes, cb, sc, x))
    rows = np.unique(np.concatenate([[0, 11007], np.random.default_rng(3).integers(0, 11008, 40)]))
    check_products(lay, y, rows)


@pytest.mark.parametrize("d_out,d_in,M,B,n", [
    (11000, 1024, 4, 8, 500),   # 128 x 256 tiles, ragged tokens and rows
    (11000, 64, 2, 8, 500),     # 128 x 256 tiles, one K-step (fewer steps than stages)
    (11000, 576, 2, 8, 1000),   # 256 x 192 tiles
    (8000, 512, 1, 16, 2000),   # 256 x 256 tiles
    (8100, 192, 2, 8, 1900),    # 256 x 256 tiles, three K-steps
    (11000, 64, 4, 8, 1030),    # 256 x 256 tiles, one K-step
])
def test_gemm_workspace_tile_shapes(d_out, d_in, M, B, n):
    """The dense product's larger tile shapes (chosen by tile count on a
    256-CU GPU), with ragged edges: every token against the oracle on sampled
    rows around the tile boundaries, and a second call bit for bit."""
    print(f"[gemm-ws tiles] {d_out}x{d_in} M={M} B={B} n={n}", flush=True)
    lay = synth.layer(8400 + d_out + d_in + n, d_out, d_in, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    y1 = aq().gemm(codes, cb, sc, x)
    y2 = aq().gemm(codes, cb, sc, x)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    edges = [0, 127, 128, 191, 192, 255, 256, d_out - 257, d_out - 256, d_out - 1]
    rows = np.unique(np.concatenate([edges, np.random.default_rng(d_out + n).integers(0, d_out, 30)]))
    check_products(lay, fp16_to_np(y1), rows)


@pytest.mark.parametrize("d_out,d_in,M,B,n", [(300, 1040, 2, 8, 63), (300, 1040, 4, 8, 200), (200, 1024, 2, 8, 16)])
def test_gemm_without_workspace_is_small_batch(d_out, d_in, M, B, n):
    """When the size query says 0 the call is exactly aqlm_gemm_small_batch
    (bit for bit) and takes no workspace."""
    lay = synth.layer(8300 + d_in + n, d_out, d_in, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    assert aq().gemm_workspace_bytes(codes, cb, sc, n) == 0
    y1 = aq().gemm(codes, cb, sc, x).cpu().numpy().view(np.uint16)
    y2 = aq().gemm_small_batch(codes, cb, sc, x).cpu().numpy().view(np.uint16)
    assert np.array_equal(y1, y2)


def test_gemm_workspace_deterministic():
    lay = synth.layer(16, 700, 2048, 2, 8, n=300)
    codes, cb, sc, x = to_device(lay)
    ys = torch.stack([aq().gemm(codes, cb, sc, x) for _ in range(100)]).cpu().numpy().view(np.uint16)
    assert (ys == ys[0]).all()


def test_gemm_small_batch_deterministic():
    lay = synth.layer(14, 3000, 4096, 4, 8, n=8)
    codes, cb, sc, x = to_device(lay)
    ys = torch.stack([aq().gemm_small_batch(codes, cb, sc, x) for _ in range(100)]).cpu().numpy().view(np.uint16)
    assert (ys == ys[0]).all()


def test_gemm_deterministic():
    lay = synth.layer(12, 2048, 2048, 2, 8, n=37)
    codes, cb, sc, x = to_device(lay)
    ys = torch.stack([aq().gemm_small_batch(codes, cb, sc, x) for _ in range(100)]).cpu().numpy().view(np.uint16)
    assert (ys == ys[0]).all()


# ----------------------------------------------------------------- error paths

def test_argument_errors_leave_outputs_untouched():
    lay = synth.layer(13, 64, 64, 2, 8)
    codes, cb, sc, x = to_device(lay)
    y = torch.full((64,), 7.0, dtype=torch.float16, device="cuda")
    import paper_2401_06118_amd._lib as L
    lib = L.load()
    st = lib.aqlm_gemv(codes.data_ptr(), cb.data_ptr(), sc.data_ptr(), 64, 60, 2, 8, 8, x.data_ptr(),
                       y.data_ptr(), None)
    assert st == 2
    st = lib.aqlm_gemv(codes.data_ptr(), cb.data_ptr(), sc.data_ptr(), 64, 64, 2, 8, 8, x.data_ptr() + 2,
                       y.data_ptr(), None)
    assert st == 4
    torch.cuda.synchronize()
    assert torch.all(y == 7.0)


def test_wrapper_rejects_bad_out_before_launch():
    """A caller's out tensor of the wrong dtype, shape or layout is refused
    before anything runs (the C ABI cannot check buffer sizes)."""
    lay = synth.layer(14, 64, 64, 2, 8, n=2)
    codes, cb, sc, x = to_device(lay)
    bad = [torch.zeros((63,), dtype=torch.float16, device="cuda"),
           torch.zeros((64,), dtype=torch.float32, device="cuda"),
           torch.zeros((64, 2), dtype=torch.float16, device="cuda").t()[0],
           torch.zeros((64,), dtype=torch.float16)]
    for out in bad:
        with pytest.raises(ValueError):
            aq().gemv(codes, cb, sc, x[0], out=out)
    for out in (torch.zeros((2, 63), dtype=torch.float16, device="cuda"),
                torch.zeros((64, 2), dtype=torch.float16, device="cuda").t()):
        with pytest.raises(ValueError):
            aq().gemm_small_batch(codes, cb, sc, x, out=out)
        with pytest.raises(ValueError):
            aq().gemm(codes, cb, sc, x, out=out)
    guard = torch.full((64, 65), 3.0, dtype=torch.float16, device="cuda")
    with pytest.raises(ValueError):
        aq().dequantize(codes, cb, sc, out=guard)
    torch.cuda.synchronize()
    assert torch.all(guard == 3.0)


# ------------------------------------------------------------- grouped launch

def _grouped_case(shapes, M, B, seed):
    lays = [synth.layer(seed + 31 * i, d_out, d_in, M, B) for i, (d_out, d_in) in enumerate(shapes)]
    probs, ys = [], []
    for lay in lays:
        codes, cb, sc, x = to_device(lay)
        y = torch.full((lay.d_out,), float("nan"), dtype=torch.float16, device="cuda")
        probs.append((codes, cb, sc, x[0], y))
        ys.append(y)
    aq().gemv_grouped(probs)
    torch.cuda.synchronize()
    for lay, y in zip(lays, ys):
        check_products(lay, fp16_to_np(y)[None, :])
    return probs


@pytest.mark.parametrize("shapes,M,B", [
    ([(4096, 4096)] * 3, 2, 8),                        # q, k, v
    ([(11008, 4096)] * 2, 2, 8),                       # gate, up
    ([(4096, 4096)] * 3, 1, 16),
    ([(1000, 4104), (64, 512), (3000, 2048), (17, 8)], 2, 8),
    ([(1024, 8192), (1024, 8192), (8192, 8192)], 4, 8),
    ([(256, 1024)] * 8, 1, 8),
    ([(100, 520), (37, 1040)], 3, 8),                  # format without the matrix-core path
])
def test_gemv_grouped_matches_oracle(shapes, M, B):
    print(f"[grouped] {shapes} M={M} B={B}", flush=True)
    _grouped_case(shapes, M, B, 8000 + M)


def test_gemv_grouped_70b_qkv():
    """The Llama-2-70B attention projections as one grouped launch: q
    8192 x 8192, k and v 1024 x 8192 (grouped-query attention), 2x8, checked
    on sampled rows of q and every row of k and v."""
    lays = [synth.layer(8300 + i, d_out, 8192, 2, 8) for i, d_out in enumerate((8192, 1024, 1024))]
    probs, ys = [], []
    for lay in lays:
        codes, cb, sc, _ = to_device(lay)
        y = torch.full((lay.d_out,), float("nan"), dtype=torch.float16, device="cuda")
        probs.append((codes, cb, sc, to_device(lays[0])[3][0], y))
        ys.append(y)
    for lay in lays[1:]:
        lay.x = lays[0].x  # one activation vector feeds q, k and v
    aq().gemv_grouped(probs)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 8191], np.random.default_rng(3).integers(0, 8192, 96)]))
    check_products(lays[0], fp16_to_np(ys[0])[None, :], rows)
    for lay, y in zip(lays[1:], ys[1:]):
        check_products(lay, fp16_to_np(y)[None, :])


# The partial-product-table kernel (2x8, d_in a multiple of 256), asked for
# explicitly: tall layers, ragged row counts, grouped.
LUT_CASES = [
    [(60000, 256)],                      # ragged last workgroup (235 rows each)
    [(49155, 512)],                      # row count not a multiple of 4
    [(65536, 1024)],                     # 256 rows per workgroup (four quads per wave)
    [(30000, 768), (30001, 768)],        # grouped, ragged
    [(50000, 2816)],                     # 11 K-slices: odd count, ring tail
]


@pytest.mark.parametrize("shapes", LUT_CASES)
def test_gemv_partial_product_tables(shapes):
    print(f"[lut] {shapes}", flush=True)
    lays = [synth.layer(8400 + 17 * i + d_out, d_out, d_in, 2, 8) for i, (d_out, d_in) in enumerate(shapes)]
    if len(lays) > 1:
        for lay in lays[1:]:
            lay.x = lays[0].x
    probs = []
    for lay in lays:
        codes, cb, sc, _ = to_device(lay)
        y = torch.full((lay.d_out,), float("nan"), dtype=torch.float16, device="cuda")
        probs.append((codes, cb, sc, to_device(lays[0])[3][0], y))
    aq().gemv_grouped(probs, path="table")
    torch.cuda.synchronize()
    for lay, pr in zip(lays, probs):
        check_products(lay, fp16_to_np(pr[4])[None, :])


@pytest.mark.parametrize("shapes", [[(1, 256)], [(5, 512)], [(4096, 4096)] * 3, [(8192, 28672)],
                                    [(1000, 2048), (64, 256), (3000, 1024)]])
@pytest.mark.parametrize("path", ["table", "gather"])
def test_gemv_forced_path(shapes, path):
    """Either kernel family on shapes the library would give to the other:
    the table kernel with few rows per workgroup (down to one row), the
    gather kernel on tall layers."""
    if path == "gather":
        shapes = [(60000, 256)] if shapes == [(1, 256)] else shapes
    print(f"[path] {path} {shapes}", flush=True)
    lays = [synth.layer(8800 + 13 * i + d_out, d_out, d_in, 2, 8) for i, (d_out, d_in) in enumerate(shapes)]
    probs = []
    for lay in lays:
        codes, cb, sc, x = to_device(lay)
        probs.append((codes, cb, sc, x[0], torch.full((lay.d_out,), float("nan"), dtype=torch.float16,
                                                      device="cuda")))
    aq().gemv_grouped(probs, path=path)
    torch.cuda.synchronize()
    for lay, pr in zip(lays, probs):
        check_products(lay, fp16_to_np(pr[4])[None, :])


def test_gemv_table_path_refused_where_unsupported():
    lay = synth.layer(8900, 64, 520, 2, 8)
    codes, cb, sc, x = to_device(lay)
    y = torch.full((64,), 5.0, dtype=torch.float16, device="cuda")
    with pytest.raises(aq().AqlmError):
        aq().gemv_grouped([(codes, cb, sc, x[0], y)], path="table")
    torch.cuda.synchronize()
    assert torch.all(y == 5.0)


@pytest.mark.parametrize("path", ["table", "auto"])
def test_gemv_partial_product_tables_70b_gate_up(path):
    """Llama-2-70B gate and up (28672 x 8192 each) as one grouped launch
    through both kernel families; sampled rows."""
    lays = [synth.layer(8500 + i, 28672, 8192, 2, 8) for i in range(2)]
    lays[1].x = lays[0].x
    x = to_device(lays[0])[3][0]
    probs = []
    for lay in lays:
        codes, cb, sc, _ = to_device(lay)
        probs.append((codes, cb, sc, x, torch.empty(28672, dtype=torch.float16, device="cuda")))
    aq().gemv_grouped(probs, path=path)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, 2, 3, 28671], np.random.default_rng(4).integers(0, 28672, 96)]))
    for lay, pr in zip(lays, probs):
        check_products(lay, fp16_to_np(pr[4])[None, :], rows)


def test_gemv_partial_product_tables_cancelling_and_special():
    """Cancelling codebooks and special-value codebooks through the table
    kernel."""
    for lay in (synth.cancelling_layer(8600, 60000, 512, 2), synth.special_layer(8601, 60000, 256, 2, 8)):
        if not np.all(np.isfinite(lay.codebooks.astype(np.float64))):
            continue
        codes, cb, sc, x = to_device(lay)
        yt = torch.empty(lay.d_out, dtype=torch.float16, device="cuda")
        aq().gemv_grouped([(codes, cb, sc, x[0], yt)], path="table")
        y = fp16_to_np(yt)[None, :]
        w = oracle.dequantize(lay.codes, lay.codebooks, lay.scales)
        ref = oracle.matmul_f16(w, lay.x)
        fin = np.isfinite(ref[0]) & (np.abs(ref[0]) < 6.0e4)
        if lay.codebooks.max() > 1:  # special values: every finite output within its bound
            err = np.abs(y.astype(np.float64) - ref)[0][fin]
            bound = elementwise_bound(w, lay.x, ref, abs_codeword_sums(lay))[0][fin]
            assert np.all(err <= bound)
        else:
            check_products(lay, y)


def test_gemv_partial_product_tables_deterministic():
    lay = synth.layer(8700, 60000, 512, 2, 8)
    codes, cb, sc, x = to_device(lay)
    ys = torch.empty((100, 60000), dtype=torch.float16, device="cuda")
    for i in range(100):
        aq().gemv_grouped([(codes, cb, sc, x[0], ys[i])], path="table")
    ys = ys.cpu().numpy().view(np.uint16)
    assert (ys == ys[0]).all()


def test_gemv_grouped_deterministic():
    probs = _grouped_case([(4096, 4096)] * 3, 2, 8, 8100)
    first = [p[4].cpu().numpy().view(np.uint16).copy() for p in probs]
    aq().gemv_grouped(probs)
    again = [p[4].cpu().numpy().view(np.uint16) for p in probs]
    assert all(np.array_equal(a, b) for a, b in zip(first, again))


def test_gemv_grouped_error_writes_nothing():
    lay = synth.layer(8200, 64, 64, 2, 8)
    codes, cb, sc, x = to_device(lay)
    y0 = torch.full((64,), 5.0, dtype=torch.float16, device="cuda")
    y1 = torch.full((64,), 5.0, dtype=torch.float16, device="cuda")
    import paper_2401_06118_amd._lib as L
    arr = (L.GemvProblem * 2)(L.GemvProblem(codes.data_ptr(), cb.data_ptr(), sc.data_ptr(), x.data_ptr(),
                                            y0.data_ptr(), 64, 64),
                              L.GemvProblem(codes.data_ptr(), cb.data_ptr(), sc.data_ptr(), x.data_ptr(),
                                            y1.data_ptr(), 64, 60))
    assert L.load().aqlm_gemv_grouped(arr, 2, 2, 8, 8, None) == 2
    torch.cuda.synchronize()
    assert torch.all(y0 == 5.0) and torch.all(y1 == 5.0)


# -------------------------------------------------------- random shapes

def _random_format(rng):
    """(M, B): every 8-bit codebook count, or 1x16."""
    if rng.random() < 0.3:
        return 1, 16
    return int(rng.integers(1, 9)), 8


def _random_d_in(rng, top=1545):
    """d_in = 8 k up to 8 * (top - 1); 60 % of them multiples of 128, whose
    code rows are 16-byte aligned for every format (the vector-load paths)."""
    k = int(rng.integers(1, top))
    if rng.random() < 0.6:
        k = max(16, k // 16 * 16)
    return 8 * k


@pytest.mark.parametrize("seed", range(24))
def test_gemv_random_shapes(seed):
    """Seeded random layers across the dispatch branches: formats, aligned and
    unaligned code rows, every row-block / K-slice layout, and 1x16 launches
    on both sides of the codebook-chunk size threshold."""
    rng = np.random.default_rng(10_000 + seed)
    M, B = _random_format(rng)
    d_in = _random_d_in(rng)
    d_out = int(rng.integers(1, 8001 if B == 16 else 3001))
    print(f"[gemv-random] seed={seed} d_out={d_out} d_in={d_in} M={M} B={B}", flush=True)
    lay = synth.layer(11_000 + seed, d_out, d_in, M, B)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y)[None, :])


@pytest.mark.parametrize("seed", range(8))
def test_gemv_grouped_random_shapes(seed):
    """Seeded random groups of 1..8 problems sharing (M, B)."""
    rng = np.random.default_rng(12_000 + seed)
    M, B = _random_format(rng)
    count = int(rng.integers(1, 9))
    shapes = [(int(rng.integers(1, 2501)), _random_d_in(rng, 1025)) for _ in range(count)]
    print(f"[grouped-random] seed={seed} M={M} B={B} {shapes}", flush=True)
    _grouped_case(shapes, M, B, 13_000 + 97 * seed)


@pytest.mark.parametrize("seed", range(16))
def test_gemm_random_shapes(seed):
    """Seeded random products with n activation rows through both entry
    points (the fused small-batch / prefill kernels and the workspace path)."""
    rng = np.random.default_rng(14_000 + seed)
    M, B = _random_format(rng)
    d_in = _random_d_in(rng, 385)                         # up to 3072
    d_out = int(rng.integers(1, 1201))
    n = int(rng.integers(2, 161))
    print(f"[gemm-random] seed={seed} n={n} d_out={d_out} d_in={d_in} M={M} B={B}", flush=True)
    lay = synth.layer(15_000 + seed, d_out, d_in, M, B, n=n)
    codes, cb, sc, x = to_device(lay)
    y1 = aq().gemm_small_batch(codes, cb, sc, x)
    y2 = aq().gemm(codes, cb, sc, x)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y1))
    check_products(lay, fp16_to_np(y2))


# ------------------------------------------------- gradients through Eq. 2

BACKWARD_CASES = [
    # (d_out, d_in, M, n)
    (64, 256, 2, 32),
    (200, 520, 1, 37),       # ragged tokens and inputs, d_out not a multiple of 128
    (1000, 1040, 4, 64),
    (1024, 4096, 2, 128),    # Llama-2-7B input width
    (96, 384, 3, 5), (40, 128, 5, 9), (16, 64, 6, 1), (8, 8, 7, 3), (136, 264, 8, 70),
]


def _backward_check(lay, dy, dcb, ds):
    ref_cb, ref_ds = oracle.backward(lay.codes, lay.codebooks, lay.scales, lay.x, dy)
    got_cb = dcb.double().cpu().numpy()
    got_ds = ds.double().cpu().numpy()
    assert rel_l2(got_cb, ref_cb) <= 1e-4, rel_l2(got_cb, ref_cb)
    assert rel_l2(got_ds, ref_ds) <= 1e-4, rel_l2(got_ds, ref_ds)
    assert np.max(np.abs(got_cb - ref_cb)) <= 1e-4 * np.max(np.abs(ref_cb))
    assert np.max(np.abs(got_ds - ref_ds)) <= 1e-4 * np.max(np.abs(ref_ds))


@pytest.mark.parametrize("d_out,d_in,M,n", BACKWARD_CASES)
def test_backward_matches_oracle(d_out, d_in, M, n):
    print(f"[backward] d_out={d_out} d_in={d_in} M={M} n={n}", flush=True)
    lay = synth.layer(20000 + d_out + d_in + M, d_out, d_in, M, 8, n=n)
    dy = np.random.default_rng(20001 + n).standard_normal((n, d_out)).astype(np.float16)
    codes, cb, sc, x = to_device(lay)
    dcb, ds = aq().backward(codes, cb, sc, x, torch.from_numpy(dy).cuda())
    torch.cuda.synchronize()
    _backward_check(lay, dy, dcb, ds)


def test_backward_accumulates_and_cancelling():
    """Two calls add up (micro-batch accumulation); codebooks that cancel in
    pairs give the same gradients as the oracle."""
    lay = synth.cancelling_layer(20100, 256, 512, 4, n=48)
    dy = np.random.default_rng(20101).standard_normal((48, 256)).astype(np.float16)
    codes, cb, sc, x = to_device(lay)
    dyt = torch.from_numpy(dy).cuda()
    dcb, ds = aq().backward(codes, cb, sc, x, dyt)
    aq().backward(codes, cb, sc, x, dyt, dcodebooks=dcb, dscales=ds)
    torch.cuda.synchronize()
    _backward_check(lay, dy, dcb / 2, ds / 2)


def test_backward_refuses_before_launch():
    lay = synth.layer(20200, 64, 256, 2, 8, n=4)
    codes, cb, sc, x = to_device(lay)
    dy = torch.zeros((4, 64), dtype=torch.float16, device="cuda")
    with pytest.raises(ValueError):
        aq().backward(codes, cb, sc, x, dy[:3])
    lay16 = synth.layer(20201, 64, 256, 1, 16, n=4)
    c16, cb16, sc16, x16 = to_device(lay16)
    with pytest.raises(aq().AqlmError):
        aq().backward(c16, cb16, sc16, x16, dy)


# ----------------------------------------------------- Phase 1: beam search

BEAM_CASES = [
    # (d_out, d_in, M, beam, sweeps)
    (16, 64, 2, 4, 2),
    (32, 128, 1, 1, 1),
    (24, 256, 3, 8, 1),
    (8, 512, 2, 2, 1),
    (40, 1024, 2, 4, 1),
    (6, 2048, 1, 8, 1),     # the largest state for beam 8
]


def _beam_inputs(seed, d_out, d_in, M, n_x=64):
    rng = np.random.default_rng(seed)
    lay = synth.layer(seed, d_out, d_in, M, 8)
    x = rng.integers(-3, 4, size=(d_in, n_x)).astype(np.float32)  # X X^T exact in fp32
    h = (x.astype(np.float64) @ x.T.astype(np.float64)).astype(np.float32)
    w = (rng.standard_normal((d_out, d_in)) * 0.05).astype(np.float32)
    return lay, w, h


@pytest.mark.parametrize("d_out,d_in,M,beam,sweeps", BEAM_CASES)
def test_beam_search_matches_oracle(d_out, d_in, M, beam, sweeps):
    """The GPU search scores candidates with fp32 increments, the oracle in
    fp64, so a near-tie can go either way and the paths may then part: most
    rows must end on exactly the oracle's codes, every row within 2e-3 of the
    oracle's loss, never above its starting loss, and the reported loss must
    be the exact loss of the returned codes."""
    print(f"[beam] d_out={d_out} d_in={d_in} M={M} beam={beam} sweeps={sweeps}", flush=True)
    lay, w, h = _beam_inputs(30000 + d_in + M + beam, d_out, d_in, M)
    ref_codes, ref_loss = oracle.beam_search(w, h, lay.codes, lay.codebooks, lay.scales, beam=beam, sweeps=sweeps)
    codes, cb, sc, _ = to_device(lay)
    loss = aq().beam_search(torch.from_numpy(w).cuda(), torch.from_numpy(h).cuda(), codes, cb, sc, beam=beam,
                            sweeps=sweeps)
    torch.cuda.synchronize()
    got = codes.cpu().numpy()
    got_loss = loss.double().cpu().numpy()
    exact = oracle.aq_loss(w, h, got, lay.codebooks, lay.scales)
    np.testing.assert_allclose(got_loss, exact, rtol=1e-6)
    np.testing.assert_allclose(exact, ref_loss, rtol=2e-3)
    differ = np.flatnonzero((got != ref_codes).any(axis=(1, 2)))
    print(f"[beam] rows with other codes than the oracle: {differ.size} of {d_out}", flush=True)
    assert differ.size <= max(1, d_out // 4), differ
    start = oracle.aq_loss(w, h, lay.codes, lay.codebooks, lay.scales)
    assert np.all(exact <= start * (1 + 1e-6))


def test_beam_search_refuses_before_launch():
    lay, w, h = _beam_inputs(30100, 8, 4096, 2)
    codes, cb, sc, _ = to_device(lay)
    before = codes.clone()
    with pytest.raises(aq().AqlmError):          # beam 8 x 4096 inputs: state beyond the on-chip budget
        aq().beam_search(torch.from_numpy(w).cuda(), torch.from_numpy(h).cuda(), codes, cb, sc, beam=8)
    torch.cuda.synchronize()
    assert torch.equal(codes, before)


# -------------------------------------------------- 1x15 (15-bit codes)

@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (11008, 4096), (4096, 11008), (1000, 4104), (37, 8)])
def test_1x15_gemv_matches_oracle(d_out, d_in):
    """One codebook of 2^15 codewords, codes stored as uint16 (the unpacked
    reading): the L2-gather and the chunked kernels (four chunks), aligned
    and unaligned code rows."""
    print(f"[1x15 gemv] {d_out}x{d_in}", flush=True)
    lay = synth.layer(16_000 + d_out + d_in, d_out, d_in, 1, 15)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y)[None, :])


def test_1x15_grouped_matches_oracle():
    _grouped_case([(4096, 4096)] * 3, 1, 15, 16_100)
    _grouped_case([(11008, 4096)] * 2, 1, 15, 16_200)


@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (1000, 4104)])
def test_1x15_dequantize_bit_exact(d_out, d_in):
    lay = synth.layer(16_300 + d_out, d_out, d_in, 1, 15)
    assert_bits_equal(dequant_gpu(lay), oracle.dequantize(lay.codes, lay.codebooks, lay.scales))


@pytest.mark.parametrize("n", [4, 16, 32, 100, 300])
def test_1x15_gemm_matches_oracle(n):
    """Small batch (chunks of 16), the tiled and prefill kernels, and the
    workspace path."""
    print(f"[1x15 gemm] n={n}", flush=True)
    lay = synth.layer(16_400 + n, 1100, 2048, 1, 15, n=n)
    codes, cb, sc, x = to_device(lay)
    y1 = aq().gemm_small_batch(codes, cb, sc, x)
    y2 = aq().gemm(codes, cb, sc, x)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y1))
    check_products(lay, fp16_to_np(y2))


def test_1x15_high_code_bits_are_ignored():
    """Codes are taken modulo 2^15: setting bit 15 of every code changes
    nothing (no codeword outside the 2^15-entry codebook is read)."""
    lay = synth.layer(16_500, 512, 1024, 1, 15)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    w = aq().dequantize(codes, cb, sc)
    high = (codes.view(torch.int16) | torch.tensor(-32768, dtype=torch.int16, device="cuda")).contiguous()
    y_hi = aq().gemv(high, cb, sc, x[0])
    w_hi = aq().dequantize(high, cb, sc)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y_hi.view(torch.int16))
    assert torch.equal(w.view(torch.int16), w_hi.view(torch.int16))


# ------------------------------- two codebooks of 12-, 15- and 16-bit codes
# (the 3- and 4-bit settings of the appendix "Experimental Configurations";
# codes stored one per uint16, m fastest)

@pytest.mark.parametrize("B", [12, 15, 16])
@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (11008, 4096), (4096, 11008), (1000, 4104), (37, 8),
                                        (64, 16384), (24, 65544)])
def test_2xwide_gemv_matches_oracle(B, d_out, d_in):
    """The matrix-core kernel with the codebooks in LDS (2x12 up to d_in =
    11008) or gathered from L2 (2x15, 2x16, and 2x12 at d_in = 16384, where x
    leaves no room for them), aligned and unaligned code rows; for d_in past
    its x staging, the vector-ALU kernel."""
    print(f"[2x{B} gemv] {d_out}x{d_in}", flush=True)
    lay = synth.layer(17_000 + 100 * B + d_out + d_in, d_out, d_in, 2, B)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y)[None, :])


@pytest.mark.parametrize("B", [12, 16])
def test_2xwide_grouped_matches_oracle(B):
    _grouped_case([(4096, 4096), (1024, 4096), (1024, 4096)], 2, B, 17_500 + B)
    _grouped_case([(11008, 4096)] * 2, 2, B, 17_600 + B)


@pytest.mark.parametrize("B", [12, 15, 16])
@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (1000, 4104)])
def test_2xwide_dequantize_bit_exact(B, d_out, d_in):
    lay = synth.layer(17_700 + B + d_out, d_out, d_in, 2, B)
    assert_bits_equal(dequant_gpu(lay), oracle.dequantize(lay.codes, lay.codebooks, lay.scales))


def test_2x12_dequantize_special_values_bit_exact():
    """Subnormals, ties, signed zeros and overflow through the fp32 sum of two
    codewords and the scale."""
    lay = synth.special_layer(17_800, 300, 1024, 2, 12)
    assert_bits_equal(dequant_gpu(lay), oracle.dequantize(lay.codes, lay.codebooks, lay.scales))


@pytest.mark.parametrize("B", [12, 15, 16])
@pytest.mark.parametrize("n", [4, 16, 32, 100, 200, 300])
def test_2xwide_gemm_matches_oracle(B, n):
    """Small batch (chunks of 16), the tiled kernel, the prefill kernel with
    two codebooks gathered from L2 (from 96 rows, 192 for 2x12; ragged row
    and token tiles) and the workspace path."""
    print(f"[2x{B} gemm] n={n}", flush=True)
    lay = synth.layer(17_900 + B + n, 1100, 2048, 2, B, n=n)
    codes, cb, sc, x = to_device(lay)
    y1 = aq().gemm_small_batch(codes, cb, sc, x)
    y2 = aq().gemm(codes, cb, sc, x)
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y1))
    check_products(lay, fp16_to_np(y2))


@pytest.mark.parametrize("B", [12, 16])
def test_2xwide_prefill_layer_sampled_rows(B):
    """11008 x 4096 with 2048 rows through the prefill kernel (256-token
    tiles, every XCD), rows sampled."""
    print(f"[2x{B} prefill] n=2048", flush=True)
    lay = synth.layer(18_100 + B, 11008, 4096, 2, B, n=2048)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemm_small_batch(codes, cb, sc, x)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 127, 128, 5503, 11006, 11007] + list(range(300, 11008, 1499)))
    check_products(lay, fp16_to_np(y), rows=rows)


def test_2x12_high_code_bits_are_ignored():
    """Codes are taken modulo 2^12: setting bits 12-15 of every code changes
    nothing (no codeword outside a 4096-entry codebook is read)."""
    lay = synth.layer(18_000, 512, 1024, 2, 12, n=4)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    yb = aq().gemm_small_batch(codes, cb, sc, x)
    w = aq().dequantize(codes, cb, sc)
    high = (codes.view(torch.int16) | torch.tensor(-4096, dtype=torch.int16, device="cuda")).contiguous()
    y_hi = aq().gemv(high, cb, sc, x[0])
    yb_hi = aq().gemm_small_batch(high, cb, sc, x)
    w_hi = aq().dequantize(high, cb, sc)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y_hi.view(torch.int16))
    assert torch.equal(yb.view(torch.int16), yb_hi.view(torch.int16))
    assert torch.equal(w.view(torch.int16), w_hi.view(torch.int16))


# ------------------------------------------------ bit-packed 12- and 15-bit codes
# (the code storage the paper's bits-per-parameter figures count: each row a
# bit string of its d_in/8 * M codes, padded to whole 32-bit words)

from paper_2401_06118_amd import format as aqfmt  # noqa: E402

PACKED_FORMATS = [(2, 12), (2, 15), (1, 15)]


def packed_device(lay):
    """(int32 packed words, codebooks, scales, x) on the GPU; the words are
    written by format.pack_codes on the host."""
    _, cb, sc, x = to_device(lay)
    B = int(lay.codebooks.shape[1]).bit_length() - 1
    words = aqfmt.pack_codes(lay.codes, B).view(np.int32)
    return torch.from_numpy(np.ascontiguousarray(words)).cuda(), cb, sc, x


@pytest.mark.parametrize("M,B", PACKED_FORMATS)
@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (1000, 4104), (37, 8), (33, 8008), (5, 11008)])
def test_packed_dequantize_bit_exact(M, B, d_out, d_in):
    """Row bit strings whose groups straddle 32-bit words (15-bit codes) and
    rows that end inside a word (ragged G * M * B)."""
    print(f"[packed dequant] {M}x{B} {d_out}x{d_in}", flush=True)
    lay = synth.layer(19_000 + 7 * B + d_out + d_in, d_out, d_in, M, B)
    words, cb, sc, _ = packed_device(lay)
    w = aq().dequantize(words, cb, sc, d_in=d_in)
    torch.cuda.synchronize()
    assert_bits_equal(w.cpu().numpy().view(np.uint16),
                      oracle.dequantize_packed(aqfmt.pack_codes(lay.codes, B), lay.codebooks, lay.scales, d_in, B),
                      "packed dequantize")


@pytest.mark.parametrize("M,B", PACKED_FORMATS)
@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (11008, 4096), (4096, 11008), (1000, 4104), (37, 8),
                                        (33, 8008), (4000, 8008), (64, 16384), (24, 65536)])
def test_packed_gemv_matches_oracle(M, B, d_out, d_in):
    """The matrix-core kernel reading packed rows: 2x12 with the codebooks in
    LDS (d_in up to 11008) and from L2, 2x15 from L2, 1x15 from L2 (small
    launches) or through LDS chunk by chunk (the 11008 x 4096, 4096 x 11008
    and 4000 x 8008 layers); ragged rows,
    slots whose codes straddle words, and the largest x the kernel stages
    (d_in = 65536; beyond it packed codes are refused).  Where the unpacked
    codes take the same kernel (two codebooks, 16-byte code rows) the result
    is bit for bit the unpacked one."""
    print(f"[packed gemv] {M}x{B} {d_out}x{d_in}", flush=True)
    lay = synth.layer(19_500 + 7 * B + d_out + d_in, d_out, d_in, M, B)
    words, cb, sc, x = packed_device(lay)
    y = aq().gemv(words, cb, sc, x[0])
    codes, _, _, _ = to_device(lay)
    y_unpacked = aq().gemv(codes, cb, sc, x[0])
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y)[None, :])
    if M == 2 and ((d_in // 8) * M * 2) % 16 == 0:
        assert torch.equal(y.view(torch.int16), y_unpacked.view(torch.int16))


@pytest.mark.parametrize("M,B", PACKED_FORMATS)
def test_packed_gemv_grouped_matches_oracle(M, B):
    """q, k, v-shaped problems and a ragged one in one grouped launch."""
    print(f"[packed grouped] {M}x{B}", flush=True)
    shapes = [(4096, 4096), (1024, 4096), (1024, 4096), (77, 4104)] if M == 2 else \
        [(4096, 4096), (300, 8008), (11008, 4096)]
    lays = [synth.layer(20_000 + 13 * i + B, o, i_, M, B) for i, (o, i_) in enumerate(shapes)]
    probs, ys = [], []
    for lay in lays:
        words, cb, sc, x = packed_device(lay)
        y = torch.empty(lay.codes.shape[0], dtype=torch.float16, device="cuda")
        probs.append((words, cb, sc, x[0], y))
        ys.append(y)
    aq().gemv_grouped(probs)
    torch.cuda.synchronize()
    for lay, y in zip(lays, ys):
        check_products(lay, fp16_to_np(y)[None, :])


def test_packed_gemv_deterministic():
    lay = synth.layer(20_100, 2048, 4096, 2, 15)
    words, cb, sc, x = packed_device(lay)
    ys = [aq().gemv(words, cb, sc, x[0]).clone() for _ in range(10)]
    torch.cuda.synchronize()
    assert all(torch.equal(ys[0].view(torch.int16), y.view(torch.int16)) for y in ys[1:])


def test_packed_codes_refused_where_unsupported():
    """Entry points without a packed path refuse before launching; so do the
    table path and aqlm_gemv when x does not fit the matrix-core kernel."""
    lay = synth.layer(20_200, 64, 1024, 2, 12, n=4)
    words, cb, sc, x = packed_device(lay)
    for fn in (lambda: aq().gemm_small_batch(words, cb, sc, x),
               lambda: aq().gemm(words, cb, sc, x)):
        with pytest.raises((ValueError, aq().AqlmError)):
            fn()
    y = torch.zeros(64, dtype=torch.float16, device="cuda")
    with pytest.raises(aq().AqlmError):
        aq().gemv_grouped([(words, cb, sc, x[0], y)], path="table")
    big = synth.layer(20_300, 4, 8 * 16400, 1, 15)
    words, cb, sc, x = packed_device(big)
    y = torch.zeros(4, dtype=torch.float16, device="cuda")
    with pytest.raises(aq().AqlmError):
        aq().gemv(words, cb, sc, x[0], out=y)
    torch.cuda.synchronize()
    assert not y.any()


# ------------------------------------------- decode step (one persistent launch)

def _step_layer(seed, d_out, d_in, x=None):
    """A 2x8 layer on the GPU with its host copy; x: a GPU fp16 vector to
    read instead of the layer's own (an earlier level's output)."""
    lay = synth.layer(seed, d_out, d_in, 2, 8)
    codes, cb, sc, xd = to_device(lay)
    y = torch.full((d_out,), float("nan"), dtype=torch.float16, device="cuda")
    return lay, (codes, cb, sc, xd[0] if x is None else x, y)


def _grouped_reference(levels):
    """The same levels as separate grouped launches, one per level, into
    fresh outputs (kernel boundaries order them)."""
    outs = []
    for lv in levels:
        ys = [torch.full_like(p[4], float("nan")) for p in lv]
        aq().gemv_grouped([(p[0], p[1], p[2], p[3], y) for p, y in zip(lv, ys)])
        outs.append(ys)
    torch.cuda.synchronize()
    return outs


def test_decode_step_chained_levels_match_oracle():
    """Level 1 reads level 0's output and level 2 level 1's: the step must
    order the levels across the whole grid.  Each output is checked against
    the oracle run through the same chain (its own fp16-rounded outputs as the
    next inputs), within the elementwise bound plus the effect of the
    previous level's bound through |W|; and bit for bit against the same
    levels launched one by one with aqlm_gemv_grouped."""
    print("[step] chained levels", flush=True)
    lay0, p0 = _step_layer(21_000, 4096, 4096)
    lay1, p1 = _step_layer(21_001, 2048, 4096, x=p0[4])
    lay2, p2 = _step_layer(21_002, 1024, 4096, x=p0[4])
    lay3, p3 = _step_layer(21_003, 4096, 2048, x=p1[4])
    levels = [[p0], [p1, p2], [p3]]
    step = aq().DecodeStep(levels)
    step.run()
    step.status()
    # oracle chain: x of a level = the oracle's fp16-rounded output of the previous one
    def run_oracle(lay, x_f16, err_in):
        w = oracle.dequantize(lay.codes, lay.codebooks, lay.scales)
        ref = oracle.matmul_f16(w, x_f16[None, :])[0]
        absw = abs_codeword_sums(lay)
        bound = elementwise_bound(w, x_f16[None, :], ref[None, :], absw)[0]
        if err_in is not None:
            bound = bound * 1.01 + np.abs(w.view(np.float16).astype(np.float64)) @ err_in
        return ref, bound
    ref0, b0 = run_oracle(lay0, lay0.x[0], None)
    x1 = ref0.astype(np.float16)
    e0 = b0 + np.abs(ref0 - x1.astype(np.float64))
    ref1, b1 = run_oracle(lay1, x1, e0)
    ref2, b2 = run_oracle(lay2, x1, e0)
    x3 = ref1.astype(np.float16)
    e1 = b1 + np.abs(ref1 - x3.astype(np.float64))
    ref3, b3 = run_oracle(lay3, x3, e1)
    for name, (p, ref, bound) in {"l0": (p0, ref0, b0), "l1a": (p1, ref1, b1), "l1b": (p2, ref2, b2),
                                  "l2": (p3, ref3, b3)}.items():
        got = fp16_to_np(p[4]).astype(np.float64)
        assert np.all(np.isfinite(got)), name
        assert rel_l2(got, ref) <= TOL, (name, rel_l2(got, ref))
        worst = int(np.argmax(np.abs(got - ref) - bound))
        assert np.all(np.abs(got - ref) <= bound), (name, worst, abs(got[worst] - ref[worst]), bound[worst])
    # the same chain, one grouped launch per level (level l's y feeds level l + 1)
    y0 = torch.empty_like(p0[4])
    y1 = torch.empty_like(p1[4])
    y2 = torch.empty_like(p2[4])
    y3 = torch.empty_like(p3[4])
    aq().gemv_grouped([(p0[0], p0[1], p0[2], p0[3], y0)])
    aq().gemv_grouped([(p1[0], p1[1], p1[2], y0, y1), (p2[0], p2[1], p2[2], y0, y2)])
    aq().gemv_grouped([(p3[0], p3[1], p3[2], y1, y3)])
    torch.cuda.synchronize()
    for a, b in ((p0[4], y0), (p1[4], y1), (p2[4], y2), (p3[4], y3)):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def _block_levels(seed, shapes, blocks):
    """Decode-step levels of `blocks` transformer blocks with the given
    projection shapes (q, k, v, o, gate, up, down), independent inputs:
    grouped q/k/v, o, grouped gate/up, down."""
    levels, lays = [], []
    for b in range(blocks):
        made = [_step_layer(seed + 16 * b + i, o, i_) for i, (o, i_) in enumerate(shapes)]
        lays += [m[0] for m in made]
        ps = [m[1] for m in made]
        x_attn, x_mlp = ps[0][3], ps[4][3]
        ps = [(c, cb, s, x_attn if i in (1, 2) else (x_mlp if i == 5 else x), y)
              for i, (c, cb, s, x, y) in enumerate(ps)]
        levels += [[ps[0], ps[1], ps[2]], [ps[3]], [ps[4], ps[5]], [ps[6]]]
    return levels, lays


def test_decode_step_7b_blocks_match_grouped_launches_and_oracle():
    """Two Llama-2-7B blocks (8 levels) in one launch: every output bit for
    bit the grouped launches' (same work split, same arithmetic), and
    sampled rows of each against the oracle."""
    print("[step] 7B blocks", flush=True)
    shapes = [(4096, 4096)] * 4 + [(11008, 4096)] * 2 + [(4096, 11008)]
    levels, lays = _block_levels(22_000, shapes, 2)
    step = aq().DecodeStep(levels)
    step.run()
    step.status()
    ref = _grouped_reference(levels)
    flat = [p for lv in levels for p in lv]
    flat_ref = [y for ys in ref for y in ys]
    for p, y in zip(flat, flat_ref):
        assert torch.equal(p[4].view(torch.int16), y.view(torch.int16))
    # lays are in shape order per block; the problems in level order are
    # q, k, v, o, gate, up, down as well
    rows = np.array([0, 1, 15, 16, 1000, 2047, 4095])
    for lay, p in zip(lays, flat):
        r = rows[rows < lay.d_out]
        x = p[3].cpu().numpy().view(np.uint16)[None, :]
        w = oracle.dequantize_rows(lay.codes, lay.codebooks, lay.scales, r)
        want = oracle.matmul_f16(w, x)
        got = fp16_to_np(p[4])[None, r].astype(np.float64)
        bound = elementwise_bound(w, x, want, abs_codeword_sums(lay, r))
        assert np.all(np.abs(got - want) <= bound)


def test_decode_step_reruns_are_identical():
    """The counters are left zero by each launch: five runs in a row, each
    status clean, all outputs identical."""
    levels, _ = _block_levels(23_000, [(1024, 1024)] * 4 + [(2816, 1024)] * 2 + [(1024, 2816)], 3)
    step = aq().DecodeStep(levels)
    outs = []
    for _ in range(5):
        for lv in levels:
            for p in lv:
                p[4].fill_(float("nan"))
        step.run()
        step.status()
        outs.append([p[4].clone() for lv in levels for p in lv])
    for o in outs[1:]:
        assert all(torch.equal(a.view(torch.int16), b.view(torch.int16)) for a, b in zip(outs[0], o))
    assert int(step.sync[0]) == 0 and int(step.sync[2]) == 0


def test_decode_step_barrier_timeout_is_reported_and_recovers():
    """A bounded wait that gives up: level 0 pairs a large layer with a
    16-row one, so the workgroup of the small one reaches level 1's barrier
    long before the others finish; with one poll allowed it times out.  The
    flag is reported (AQLM_ERR_TIMEOUT), level 1 is left unwritten, the
    launch ends normally, and the next run with the default limit computes
    everything."""
    print("[step] timeout", flush=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(24_000)
    big = synth.device_layer(24_001, 28672, 8192, 2, 8)
    small = synth.device_layer(24_002, 16, 8192, 2, 8)
    nxt = synth.device_layer(24_003, 4096, 4096, 2, 8)
    ys = [torch.full((d,), float("nan"), dtype=torch.float16, device="cuda") for d in (28672, 16, 4096)]
    levels = [[(big[0], big[1], big[2], big[3][0], ys[0]), (small[0], small[1], small[2], small[3][0], ys[1])],
              [(nxt[0], nxt[1], nxt[2], nxt[3][0], ys[2])]]
    step = aq().DecodeStep(levels)
    step.run(spin_limit=1)
    with pytest.raises(aq().AqlmError) as e:
        step.status()
    assert e.value.status == 8
    assert torch.isnan(ys[2].float()).all()          # level 1 never ran
    assert int(step.sync[0]) == 0 and int(step.sync[2]) == 0   # counters reset by the last workgroup out
    step.run()
    step.status()
    ref = _grouped_reference(levels)
    for got, want in zip(ys, [y for r in ref for y in r]):
        assert torch.equal(got.view(torch.int16), want.view(torch.int16))


def test_decode_step_refuses_other_formats():
    lay = synth.layer(25_000, 64, 1024, 4, 8)
    codes, cb, sc, x = to_device(lay)
    y = torch.empty(64, dtype=torch.float16, device="cuda")
    with pytest.raises(aq().AqlmError):
        aq().DecodeStep([[(codes, cb, sc, x[0], y)]])


# ------------------------------ larger groups (codebooks-versus-groups ablation)
# 4x8 with groups of 16, 8x8 with 32, 15x8 with 64 (about two bits per weight)

GROUP_FORMATS = [(4, 16), (8, 32), (15, 64)]


@pytest.mark.parametrize("M,g", GROUP_FORMATS + [(1, 16), (3, 32), (16, 64)])
@pytest.mark.parametrize("d_out,d_in", [(300, 1024), (37, 192), (1, 64), (1000, 4096)])
def test_large_groups_dequantize_bit_exact(M, g, d_out, d_in):
    print(f"[groups dequant] {M}x8 g{g} {d_out}x{d_in}", flush=True)
    lay = synth.layer(26_000 + M + g + d_out, d_out, d_in, M, 8, g=g)
    assert_bits_equal(dequant_gpu(lay), oracle.dequantize(lay.codes, lay.codebooks, lay.scales, g),
                      "large-group dequantize")


def test_large_groups_dequantize_special_values_bit_exact():
    lay = synth.special_layer(26_100, 129, 256, 4, 8, g=16)
    ref = oracle.dequantize(lay.codes, lay.codebooks, lay.scales, 16)
    assert_bits_equal(dequant_gpu(lay), ref, "large-group dequantize special")
    assert np.any(ref == 0x8000) and np.any((ref & 0x7C00) == 0)


@pytest.mark.parametrize("M,g", GROUP_FORMATS)
@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (11008, 4096), (4096, 11008), (37, 192)])
def test_large_groups_gemv_matches_oracle(M, g, d_out, d_in):
    """Codebooks in LDS (4x8 gs16 32 KiB, 8x8 gs32 128 KiB) or gathered from
    L2 (15x8 gs64, 480 KiB); one wave per row."""
    print(f"[groups gemv] {M}x8 g{g} {d_out}x{d_in}", flush=True)
    lay = synth.layer(26_200 + M + g + d_out + d_in, d_out, d_in, M, 8, g=g)
    codes, cb, sc, x = to_device(lay)
    y = aq().gemv(codes, cb, sc, x[0])
    torch.cuda.synchronize()
    check_products(lay, fp16_to_np(y)[None, :])


@pytest.mark.parametrize("M,g", GROUP_FORMATS)
def test_large_groups_grouped_small_batch_and_workspace(M, g):
    """Grouped launches (one product per problem), n rows through the small-
    batch entry point (one product per row), and the workspace product
    (dequantize, then the dense product) at 64 and 300 rows; the no-
    allocation variant bit for bit as the workspace product."""
    print(f"[groups gemm] {M}x8 g{g}", flush=True)
    lays = [synth.layer(26_300 + M + g + i, 500 + 64 * i, 1024, M, 8, g=g) for i in range(2)]
    probs = []
    for lay in lays:
        codes, cb, sc, x = to_device(lay)
        probs.append((codes, cb, sc, x[0], torch.full((lay.d_out,), float("nan"), dtype=torch.float16,
                                                      device="cuda")))
    aq().gemv_grouped(probs)
    torch.cuda.synchronize()
    for lay, p in zip(lays, probs):
        check_products(lay, fp16_to_np(p[4])[None, :])
    for n in (3, 64, 300):
        lay = synth.layer(26_400 + M + g + n, 700, 1024, M, 8, n=n, g=g)
        codes, cb, sc, x = to_device(lay)
        y1 = aq().gemm_small_batch(codes, cb, sc, x)
        y2 = aq().gemm(codes, cb, sc, x)
        torch.cuda.synchronize()
        check_products(lay, fp16_to_np(y1))
        check_products(lay, fp16_to_np(y2))


def test_large_groups_refused_elsewhere():
    """Entry points without a large-group path refuse before launching."""
    lay = synth.layer(26_500, 64, 256, 4, 8, n=4, g=16)
    codes, cb, sc, x = to_device(lay)
    y = torch.zeros(64, dtype=torch.float16, device="cuda")
    with pytest.raises(aq().AqlmError):
        aq().gemv_grouped([(codes, cb, sc, x[0], y)], path="table")
    dcb = torch.zeros(tuple(cb.shape), dtype=torch.float32, device="cuda")
    with pytest.raises(aq().AqlmError):
        aq().backward(codes, cb, sc, x, torch.zeros((4, 64), dtype=torch.float16, device="cuda"), dcodebooks=dcb)
    w = torch.zeros((64, 256), dtype=torch.float32, device="cuda")
    h = torch.eye(256, dtype=torch.float32, device="cuda")
    with pytest.raises(aq().AqlmError):
        aq().beam_search(w, h, codes, cb, sc, beam=2)
    torch.cuda.synchronize()
    assert not y.any()
