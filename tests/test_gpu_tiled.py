"""Tiled 8-bit codes (aqlm_tile_codes, aqlm_gemv_grouped_tiled) through the C ABI.

The tiled bytes are checked against the layout written out here with numpy
(bit for bit, padding included); products over tiled codes against the
oracle (to the product tolerance) and against the row-major grouped product,
whose arithmetic they share (bit for bit).
"""
import numpy as np
import pytest

import oracle  # noqa: F401  (the parity helpers below call it)
from paper_2401_06118_amd import synth

from helpers import fp16_to_np, to_device
from test_gpu_parity import check_products

pytestmark = pytest.mark.gpu

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


def tiled_layout(codes: np.ndarray) -> np.ndarray:
    """Row-major codes [d_out, G, M] uint8 in the tiled byte order: byte c of
    row r at ((r // 16) * ks + c // 64) * 1024 + (r % 16) * 64 + c % 64, with
    ks = ceil(G * M / 64); rows past d_out and bytes past G * M zero."""
    d_out = codes.shape[0]
    row_bytes = codes.shape[1] * codes.shape[2]
    ks = -(-row_bytes // 64)
    blocks = -(-d_out // 16)
    full = np.zeros((blocks * 16, ks * 64), dtype=np.uint8)
    full[:d_out, :row_bytes] = codes.reshape(d_out, row_bytes)
    # [block, r16, ks, 64] -> [block, ks, r16, 64]
    return full.reshape(blocks, 16, ks, 64).transpose(0, 2, 1, 3).reshape(-1)


TILE_SHAPES = [(1, 8, 1), (16, 64, 2), (37, 200, 2), (1000, 4104, 2), (33, 1032, 1), (100, 520, 4),
               (8192, 8192, 2)]


@pytest.mark.parametrize("d_out,d_in,M", TILE_SHAPES)
def test_tile_codes_layout(d_out, d_in, M):
    print(f"[tile] {d_out}x{d_in} M={M}", flush=True)
    lay = synth.layer(9100 + d_out + M, d_out, d_in, M, 8)
    codes, cb, sc, _ = to_device(lay)
    t = aq().TiledCodes(codes, cb, sc)
    torch.cuda.synchronize()
    want = tiled_layout(lay.codes)
    assert t.codes.numel() == want.size
    assert np.array_equal(t.codes.cpu().numpy(), want)


# (shapes of one grouped launch, M): ragged rows and K-slices, the row-major
# unaligned-pitch class, Llama-2 7B and 70B launches
TILED_CASES = [
    ([(1, 8)], 2),                       # one row, one group: a single, mostly padded tile
    ([(1, 8), (5, 16)], 4),
    ([(37, 200)], 2),
    ([(1000, 4104), (64, 512), (3000, 2048), (17, 8)], 2),
    ([(100, 1032), (40, 520)], 2),
    ([(4096, 4096)] * 3, 2),
    ([(11008, 4096)] * 2, 2),
    ([(4096, 11008)], 2),
    ([(256, 1024)] * 8, 1),
    ([(1024, 8192), (1024, 8192), (8192, 8192)], 4),
]


def _tiled_and_row_major(shapes, M, seed):
    lays = [synth.layer(seed + 31 * i, d_out, d_in, M, 8) for i, (d_out, d_in) in enumerate(shapes)]
    row_major, tiled, ys_rm, ys_t = [], [], [], []
    for lay in lays:
        codes, cb, sc, x = to_device(lay)
        y_rm = torch.full((lay.d_out,), float("nan"), dtype=torch.float16, device="cuda")
        y_t = torch.full((lay.d_out,), float("nan"), dtype=torch.float16, device="cuda")
        row_major.append((codes, cb, sc, x[0], y_rm))
        tiled.append((aq().TiledCodes(codes, cb, sc), x[0], y_t))
        ys_rm.append(y_rm)
        ys_t.append(y_t)
    aq().gemv_grouped(row_major, path="gather")
    # Row-major problems whose row pitches fall in different 16-byte alignment
    # classes run as one launch each (the grouped kernel takes one class), so
    # the tiled products are launched the same way to share the row split.
    if len({(d_in // 8 * M) % 16 == 0 for _, d_in in shapes}) == 1:
        aq().gemv_tiled_grouped(tiled)
    else:
        for t in tiled:
            aq().gemv_tiled_grouped([t])
    torch.cuda.synchronize()
    return lays, ys_rm, ys_t, tiled


@pytest.mark.parametrize("shapes,M", TILED_CASES)
def test_gemv_tiled_matches_oracle_and_row_major(shapes, M):
    print(f"[tiled] {shapes} M={M}", flush=True)
    lays, ys_rm, ys_t, _ = _tiled_and_row_major(shapes, M, 9300 + M)
    for lay, y_rm, y_t in zip(lays, ys_rm, ys_t):
        got = fp16_to_np(y_t)
        rows = None
        if lay.d_out > 4096:
            rows = np.unique(np.concatenate([[0, lay.d_out - 1],
                                             np.random.default_rng(5).integers(0, lay.d_out, 96)]))
        check_products(lay, got[None, :], rows)
        assert np.array_equal(got.view(np.uint16), fp16_to_np(y_rm).view(np.uint16))


def test_gemv_tiled_70b_launches_match_row_major():
    """The Llama-2-70B launches (q/k/v grouped, o, gate/up grouped, down) on
    tiled codes equal the row-major product bit for bit; sampled rows against
    the oracle."""
    launches = [[(8192, 8192), (1024, 8192), (1024, 8192)], [(8192, 8192)], [(28672, 8192)] * 2,
                [(8192, 28672)]]
    for i, shapes in enumerate(launches):
        print(f"[tiled 70b] {shapes}", flush=True)
        lays, ys_rm, ys_t, tiled = _tiled_and_row_major(shapes, 2, 9500 + 100 * i)
        for lay, y_rm, y_t in zip(lays, ys_rm, ys_t):
            got = fp16_to_np(y_t)
            assert np.array_equal(got.view(np.uint16), fp16_to_np(y_rm).view(np.uint16))
            rows = np.unique(np.concatenate([[0, lay.d_out - 1],
                                             np.random.default_rng(7 + i).integers(0, lay.d_out, 32)]))
            check_products(lay, got[None, :], rows)
        del tiled
        torch.cuda.empty_cache()


def test_gemv_tiled_deterministic():
    lays, _, ys_t, tiled = _tiled_and_row_major([(4096, 4096)] * 3, 2, 9700)
    first = [y.cpu().numpy().view(np.uint16).copy() for y in ys_t]
    aq().gemv_tiled_grouped(tiled)
    again = [y.cpu().numpy().view(np.uint16) for y in ys_t]
    assert all(np.array_equal(a, b) for a, b in zip(first, again))


def test_tiled_errors():
    import ctypes
    import paper_2401_06118_amd._lib as L
    lib = L.load()
    lay = synth.layer(9800, 64, 256, 2, 8)
    codes, cb, sc, x = to_device(lay)
    need = int(lib.aqlm_tiled_codes_bytes(64, 256, 2, 8, 8))
    assert need == 4 * 1 * 1024
    buf = torch.zeros(need + 16, dtype=torch.uint8, device="cuda")
    # too small, misaligned, NULL, unsupported formats
    assert lib.aqlm_tile_codes(codes.data_ptr(), 64, 256, 2, 8, 8, buf.data_ptr(), need - 1, None) == 6
    assert lib.aqlm_tile_codes(codes.data_ptr(), 64, 256, 2, 8, 8, buf.data_ptr() + 1, need, None) == 4
    assert lib.aqlm_tile_codes(None, 64, 256, 2, 8, 8, buf.data_ptr(), need, None) == 1
    assert lib.aqlm_tile_codes(codes.data_ptr(), 64, 256, 2, 16, 8, buf.data_ptr(), need, None) == 3
    assert lib.aqlm_tile_codes(codes.data_ptr(), 64, 256, 3, 8, 8, buf.data_ptr(), need, None) == 3
    assert lib.aqlm_tile_codes(codes.data_ptr(), 64, 250, 2, 8, 8, buf.data_ptr(), need, None) == 2
    torch.cuda.synchronize()
    assert int(buf.sum()) == 0  # nothing written by a refused call
    t = aq().TiledCodes(codes, cb, sc)
    y = torch.full((64,), 5.0, dtype=torch.float16, device="cuda")
    arr = (L.GemvProblem * 1)(L.GemvProblem(t.codes.data_ptr(), cb.data_ptr(), sc.data_ptr(), x.data_ptr(),
                                            y.data_ptr(), 64, 256))
    assert lib.aqlm_gemv_grouped_tiled(arr, 1, 2, 16, 8, None) == 3
    assert lib.aqlm_gemv_grouped_tiled(arr, 0, 2, 8, 8, None) == 2
    assert lib.aqlm_gemv_grouped_tiled(None, 1, 2, 8, 8, None) == 1
    arr[0].x = ctypes.c_void_p(x.data_ptr() + 2).value
    assert lib.aqlm_gemv_grouped_tiled(arr, 1, 2, 8, 8, None) == 4
    torch.cuda.synchronize()
    assert torch.all(y == 5.0)
    with pytest.raises(ValueError):
        aq().TiledCodes(*to_device(synth.layer(9801, 64, 256, 1, 16))[:3])


# Small batch over tiled codes: (d_out, d_in, M, n) - ragged rows and
# K-slices, the unaligned-pitch class, 7B shapes, 1..64 rows (chunks of 16,
# a last chunk of one row).
NB_CASES = [(37, 200, 2, 2), (1000, 4104, 2, 3), (100, 1032, 4, 16), (4096, 4096, 2, 4), (11008, 4096, 4, 16),
            (4096, 11008, 2, 8), (256, 1024, 2, 1), (256, 1024, 1, 1), (300, 520, 2, 17), (1000, 1032, 4, 40),
            (512, 4096, 2, 64), (1, 8, 2, 1), (1, 8, 4, 2), (3, 16, 2, 33)]


@pytest.mark.parametrize("d_out,d_in,M,n", NB_CASES)
def test_gemm_small_batch_tiled(d_out, d_in, M, n):
    print(f"[tiled small batch] {d_out}x{d_in} M={M} n={n}", flush=True)
    lay = synth.layer(9900 + d_out + M + n, d_out, d_in, M, 8, n=n)
    codes, cb, sc, x = to_device(lay)
    y_rm = aq().gemm_small_batch(codes, cb, sc, x)
    t = aq().TiledCodes(codes, cb, sc)
    y_t = t.gemm_small_batch(x)
    torch.cuda.synchronize()
    got = fp16_to_np(y_t)
    rows = None
    if d_out > 4096:
        rows = np.unique(np.concatenate([[0, d_out - 1], np.random.default_rng(11).integers(0, d_out, 64)]))
    check_products(lay, got, rows)
    assert np.array_equal(got.view(np.uint16), fp16_to_np(y_rm).view(np.uint16))


def test_gemm_small_batch_tiled_refusals():
    lay = synth.layer(9990, 64, 256, 1, 8, n=2)
    codes, cb, sc, x = to_device(lay)
    t = aq().TiledCodes(codes, cb, sc)
    with pytest.raises(RuntimeError):
        t.gemm_small_batch(x)  # M = 1 with two rows
    lay = synth.layer(9991, 64, 256, 2, 8, n=65)
    codes, cb, sc, x = to_device(lay)
    t = aq().TiledCodes(codes, cb, sc)
    out = torch.full((65, 64), 5.0, dtype=torch.float16, device="cuda")
    with pytest.raises(RuntimeError):
        t.gemm_small_batch(x, out=out)  # more than 64 rows
    torch.cuda.synchronize()
    assert torch.all(out == 5.0)
