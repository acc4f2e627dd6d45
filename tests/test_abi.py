"""Host-side checks of the C ABI: the library loads, exports every function
include/aqlm.h declares, and rejects bad arguments before touching the GPU
(argument validation dereferences nothing, so fake pointers suffice)."""
import ctypes
import struct
import os
import re

import pytest

from paper_2401_06118_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aqlm.h")

OK, NULL, SHAPE, UNSUP, ALIGN, WORKSPACE = 0, 1, 2, 3, 4, 6
P = 0x10000  # a 64 KiB-aligned fake device address; never dereferenced on error paths


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|int64_t|size_t|const char\*)\s+(aqlm_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.skip("library not built (run python -m paper_2401_06118_amd.build)")
    return _lib.load()


def test_header_declares_the_three_operations():
    assert set(declared_functions()) >= {"aqlm_dequantize", "aqlm_gemv", "aqlm_gemm_small_batch",
                                         "aqlm_status_string"}


def test_library_exports_every_declared_function(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(_lib.EXPORTS) <= set(declared_functions())


def test_status_strings(lib):
    for st in range(7):
        assert lib.aqlm_status_string(st)
    assert lib.aqlm_status_string(99) == b"unknown status"


def gemv(lib, codes=P, cb=P, sc=P, d_out=64, d_in=64, M=2, B=8, g=8, x=P, y=P):
    return lib.aqlm_gemv(codes, cb, sc, d_out, d_in, M, B, g, x, y, None)


def gemm(lib, n=4, codes=P, cb=P, sc=P, d_out=64, d_in=64, M=2, B=8, g=8, x=P, y=P):
    return lib.aqlm_gemm_small_batch(codes, cb, sc, d_out, d_in, M, B, g, n, x, y, None)


def deq(lib, codes=P, cb=P, sc=P, d_out=64, d_in=64, M=2, B=8, g=8, w=P):
    return lib.aqlm_dequantize(codes, cb, sc, d_out, d_in, M, B, g, w, None)


def gemm_ws(lib, n=64, codes=P, cb=P, sc=P, d_out=64, d_in=64, M=2, B=8, g=8, x=P, y=P, ws=P, ws_bytes=1 << 20):
    """aqlm_gemm at n = 64 (the workspace path) - every case below fails its
    checks before anything is launched."""
    return lib.aqlm_gemm(codes, cb, sc, d_out, d_in, M, B, g, n, x, y, ws, ws_bytes, None)


@pytest.mark.parametrize("fn", [gemv, gemm, deq, gemm_ws])
def test_null_pointers(lib, fn):
    for kw in ("codes", "cb", "sc"):
        assert fn(lib, **{kw: None}) == NULL
    if fn is deq:
        assert fn(lib, w=None) == NULL
    else:
        assert fn(lib, x=None) == NULL
        assert fn(lib, y=None) == NULL


@pytest.mark.parametrize("fn", [gemv, gemm, deq, gemm_ws])
def test_shapes(lib, fn):
    assert fn(lib, d_out=0) == SHAPE
    assert fn(lib, d_out=-3) == SHAPE
    assert fn(lib, d_in=0) == SHAPE
    assert fn(lib, d_in=12) == SHAPE          # not a multiple of g
    assert fn(lib, d_out=1 << 20, d_in=1 << 14) == SHAPE  # d_out * d_in/g >= 2^31
    assert fn(lib, d_out=1, d_in=1 << 31) == SHAPE        # d_in beyond 32 bits


def test_gemm_batch_size(lib):
    assert gemm(lib, n=0) == SHAPE
    assert gemm(lib, n=-1) == SHAPE


@pytest.mark.parametrize("fn", [gemv, gemm, deq, gemm_ws])
def test_unsupported_formats(lib, fn):
    assert fn(lib, g=4, d_in=64) == UNSUP
    assert fn(lib, M=0) == UNSUP
    assert fn(lib, M=9) == UNSUP
    assert fn(lib, M=3, B=16) == UNSUP
    assert fn(lib, M=4, B=12) == UNSUP
    assert fn(lib, M=2, B=13) == UNSUP
    assert fn(lib, M=2, B=14) == UNSUP
    assert fn(lib, M=1, B=12) == UNSUP
    assert fn(lib, M=1, B=14) == UNSUP
    assert fn(lib, M=1, B=4) == UNSUP


@pytest.mark.parametrize("fn", [gemv, gemm, deq, gemm_ws])
def test_alignment(lib, fn):
    assert fn(lib, codes=P + 1) == ALIGN
    assert fn(lib, cb=P + 8) == ALIGN
    assert fn(lib, sc=P + 1) == ALIGN
    if fn is deq:
        assert fn(lib, w=P + 2) == ALIGN
    else:
        assert fn(lib, x=P + 2) == ALIGN
        assert fn(lib, y=P + 4) == ALIGN


def test_binding_refuses_cpu_tensors():
    import torch
    import paper_2401_06118_amd as aq
    codes = torch.zeros((4, 2, 2), dtype=torch.uint8)
    cb = torch.zeros((2, 256, 8), dtype=torch.float16)
    sc = torch.ones(4, dtype=torch.float16)
    with pytest.raises(ValueError):
        aq.dequantize(codes, cb, sc)


def test_grouped_validation(lib):
    Prob = _lib.GemvProblem
    good = Prob(P, P, P, P, P, 64, 64)
    arr = (Prob * 9)(*([good] * 9))
    assert lib.aqlm_gemv_grouped(None, 1, 2, 8, 8, None) == NULL
    assert lib.aqlm_gemv_grouped(arr, 0, 2, 8, 8, None) == SHAPE
    assert lib.aqlm_gemv_grouped(arr, 9, 2, 8, 8, None) == SHAPE
    assert lib.aqlm_gemv_grouped(arr, 2, 3, 16, 8, None) == UNSUP
    bad = (Prob * 3)(good, Prob(P, P, P, P, P, 64, 60), good)
    assert lib.aqlm_gemv_grouped(bad, 3, 2, 8, 8, None) == SHAPE
    bad = (Prob * 2)(good, Prob(P, P, P, None, P, 64, 64))
    assert lib.aqlm_gemv_grouped(bad, 2, 2, 8, 8, None) == NULL
    bad = (Prob * 2)(good, Prob(P, P, P, P + 2, P, 64, 64))
    assert lib.aqlm_gemv_grouped(bad, 2, 2, 8, 8, None) == ALIGN


def test_gemm_workspace(lib):
    """The workspace path: size query, and a missing, small or misaligned
    workspace is refused before anything is launched."""
    need = 64 * 64 * 2
    assert lib.aqlm_gemm_workspace_bytes(64, 64, 2, 8, 8, 64) == need
    assert lib.aqlm_gemm_workspace_bytes(64, 64, 1, 16, 8, 1000) == need
    assert lib.aqlm_gemm_workspace_bytes(11008, 4096, 4, 8, 8, 2048) == 11008 * 4096 * 2
    # few tiles (32 of 128 x 128 against 256 CUs): split along K in 8, fp32 partials after the weights
    assert lib.aqlm_gemm_workspace_bytes(4096, 11008, 4, 8, 8, 64) == 4096 * 11008 * 2 + 8 * 64 * 4096 * 4
    assert lib.aqlm_gemm_workspace_bytes(64, 64, 2, 8, 8, 63) == 0      # few rows: no workspace
    assert lib.aqlm_gemm_workspace_bytes(64, 72, 2, 8, 8, 64) == 0      # d_in not a multiple of 64
    assert lib.aqlm_gemm_workspace_bytes(0, 64, 2, 8, 8, 64) == 0       # invalid sizes
    assert lib.aqlm_gemm_workspace_bytes(64, 60, 2, 8, 8, 64) == 0
    assert lib.aqlm_gemm_workspace_bytes(64, 64, 2, 8, 8, 0) == 0
    assert gemm_ws(lib, ws=None) == NULL
    assert gemm_ws(lib, ws_bytes=need - 1) == WORKSPACE
    assert gemm_ws(lib, ws=P + 8) == ALIGN
    assert gemm_ws(lib, n=0) == SHAPE


def test_grouped_path_validation(lib):
    """aqlm_gemv_grouped_path: unknown paths, and the table path on formats or
    shapes it does not take, are refused before anything is launched."""
    Prob = _lib.GemvProblem
    good = Prob(P, P, P, P, P, 64, 64)
    arr = (Prob * 2)(good, good)
    for path in (-1, 3, 100):
        assert lib.aqlm_gemv_grouped_path(arr, 2, 2, 8, 8, path, None) == UNSUP
    assert lib.aqlm_gemv_grouped_path(arr, 2, 2, 8, 8, 2, None) == UNSUP      # d_in not a multiple of 256
    wide = (Prob * 1)(Prob(P, P, P, P, P, 64, 512))
    assert lib.aqlm_gemv_grouped_path(wide, 1, 1, 16, 8, 2, None) == UNSUP    # 1x16
    assert lib.aqlm_gemv_grouped_path(wide, 1, 4, 8, 8, 2, None) == UNSUP     # 4x8
    assert lib.aqlm_gemv_grouped_path(None, 1, 2, 8, 8, 0, None) == NULL
    bad = (Prob * 1)(Prob(P, P, P, P, P, 64, 60))
    assert lib.aqlm_gemv_grouped_path(bad, 1, 2, 8, 8, 2, None) == SHAPE


def test_noalloc_refuses_before_launch(lib):
    """aqlm_gemm_noalloc: bad arguments, and a product needing more than the
    fixed scratch buffer (AQLM_ERR_SCRATCH), are refused on the host."""
    def call(codes=P, d_out=64, d_in=64, n=64, M=2, B=8, x=P, y=P):
        return lib.aqlm_gemm_noalloc(codes, P, P, d_out, d_in, M, B, 8, n, x, y, None)
    assert call(codes=None) == NULL
    assert call(x=None) == NULL
    assert call(d_in=60) == SHAPE
    assert call(n=0) == SHAPE
    assert call(M=3, B=16) == UNSUP
    assert call(x=P + 2) == ALIGN
    assert call(d_out=12288, d_in=8192) == 7            # 192 MiB of weights
    assert call(d_out=28672, d_in=8192, n=2048) == 7
    assert lib.aqlm_status_string(7) != b"unknown status"


def test_backward_refuses_before_launch(lib):
    def call(codes=P, d_out=64, d_in=64, M=2, B=8, n=4, x=P, dy=P, dc=P, ds=P):
        return lib.aqlm_backward(codes, P, P, d_out, d_in, M, B, 8, n, x, dy, dc, ds, None)
    assert call(dc=None) == NULL
    assert call(dy=None) == NULL
    assert call(n=0) == SHAPE
    assert call(d_out=60) == SHAPE          # d_out not a multiple of 8
    assert call(M=1, B=16) == UNSUP
    assert call(M=2, B=12) == UNSUP
    assert call(dy=P + 2) == ALIGN
    assert call(ds=P + 2) == ALIGN


def test_beam_search_refuses_before_launch(lib):
    def call(w=P, h=P, codes=P, d_out=8, d_in=64, M=2, B=8, beam=4, sweeps=1, loss=P):
        return lib.aqlm_beam_search(w, h, codes, P, P, d_out, d_in, M, B, 8, beam, sweeps, loss, None)
    assert call(w=None) == NULL
    assert call(h=None) == NULL
    assert call(beam=0) == SHAPE
    assert call(sweeps=-1) == SHAPE
    assert call(M=1, B=16) == UNSUP
    assert call(beam=9) == UNSUP
    assert call(d_in=4096, beam=8) == UNSUP      # state beyond the on-chip budget
    assert call(w=P + 2) == ALIGN


PACKED = _lib.PACKED


def test_packed_row_words(lib):
    # ceil(G * M * B / 32): 2x12 -> 3 words per 4 groups, 1x15 / 2x15 ragged
    assert lib.aqlm_packed_row_words(4096, 2, 12, 8) == 4096 // 8 * 24 // 32
    assert lib.aqlm_packed_row_words(4096, 2, 12 | PACKED, 8) == 384
    assert lib.aqlm_packed_row_words(8, 1, 15, 8) == 1
    assert lib.aqlm_packed_row_words(24, 1, 15, 8) == 2
    assert lib.aqlm_packed_row_words(8008, 2, 15, 8) == (1001 * 30 + 31) // 32
    assert lib.aqlm_packed_row_words(0, 2, 12, 8) == 0


def test_packed_codes_accepted_only_where_supported(lib):
    """Packed codes: 2x12, 2x15 and 1x15 pass the checks of dequantize and
    gemv (the calls then fail only on the fake pointers' alignment); every
    other format, and every other entry point, refuses them."""
    for M, B in ((2, 12), (2, 15), (1, 15)):
        assert deq(lib, M=M, B=B | PACKED, w=P + 2) == ALIGN
        assert gemv(lib, M=M, B=B | PACKED, y=P + 2) == ALIGN
        assert gemm(lib, M=M, B=B | PACKED) == UNSUP
        assert gemm_ws(lib, M=M, B=B | PACKED) == UNSUP
    for M, B in ((2, 8), (1, 16), (2, 16), (4, 8), (1, 12)):
        assert deq(lib, M=M, B=B | PACKED) == UNSUP
        assert gemv(lib, M=M, B=B | PACKED) == UNSUP
    # x beyond the matrix-core kernel's staging: no packed fallback
    assert gemv(lib, d_in=8 * 16400, M=1, B=15 | PACKED) == UNSUP


def test_packed_codes_refused_by_other_entry_points(lib):
    p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    assert lib.aqlm_gemm_noalloc(P, P, P, 64, 64, 2, 12 | PACKED, 8, 4, P, P, None) == UNSUP
    assert lib.aqlm_backward(P, P, P, 64, 64, 2, 12 | PACKED, 8, 4, P, P, P, P, None) == UNSUP
    assert lib.aqlm_beam_search(P, P, P, P, P, 8, 64, 2, 12 | PACKED, 8, 4, 1, P, None) == UNSUP
    Prob = _lib.GemvProblem
    arr = (Prob * 1)(Prob(P, P, P, P, P, 64, 64))
    assert lib.aqlm_gemv_grouped_path(arr, 1, 2, 12 | PACKED, 8, _lib.PATH_TABLE, None) == UNSUP
    assert lib.aqlm_gemv_grouped_path(arr, 1, 2, 8 | PACKED, 8, _lib.PATH_GATHER, None) == UNSUP


def test_binding_checks_packed_shapes():
    import torch
    import paper_2401_06118_amd as aq
    cb = torch.zeros((2, 4096, 8), dtype=torch.float16)
    sc = torch.ones(4, dtype=torch.float16)
    words = torch.zeros((4, 3), dtype=torch.int32)
    with pytest.raises(ValueError):
        aq.packed_layer_args(words, cb, sc, 32)  # CPU tensors


def _step_problems(n, d_out=64, d_in=1024):
    Prob = _lib.GemvProblem
    return (Prob * n)(*[Prob(P, P, P, P, P, d_out, d_in) for _ in range(n)])


def test_decode_step_plan_on_the_host(lib):
    """A plan is built on the host without touching the GPU (the pointers are
    only recorded): header fields, size, and the refusals."""
    one = lib.aqlm_gemv_step_plan_bytes(1)
    assert one > 16 and lib.aqlm_gemv_step_plan_bytes(3) == 16 + 3 * (one - 16)
    assert lib.aqlm_gemv_step_plan_bytes(0) == 0
    sizes = (ctypes.c_int32 * 3)(3, 1, 2)
    probs = _step_problems(6)
    nbytes = lib.aqlm_gemv_step_plan_bytes(3)
    buf = ctypes.create_string_buffer(nbytes)
    assert lib.aqlm_gemv_step_plan(probs, sizes, 3, 2, 8, 8, ctypes.addressof(buf), nbytes) == OK
    magic, levels, lds, grid = struct.unpack_from("<Iiii", buf.raw)
    assert magic != 0 and levels == 3 and 0 < lds <= 160 * 1024 and grid > 0
    assert lib.aqlm_gemv_step_plan(probs, sizes, 3, 2, 8, 8, ctypes.addressof(buf), nbytes - 1) == WORKSPACE
    assert lib.aqlm_gemv_step_plan(None, sizes, 3, 2, 8, 8, ctypes.addressof(buf), nbytes) == NULL
    assert lib.aqlm_gemv_step_plan(probs, sizes, 0, 2, 8, 8, ctypes.addressof(buf), nbytes) == SHAPE
    bad = (ctypes.c_int32 * 3)(3, 0, 3)
    assert lib.aqlm_gemv_step_plan(probs, bad, 3, 2, 8, 8, ctypes.addressof(buf), nbytes) == SHAPE
    nine = (ctypes.c_int32 * 1)(9)
    assert lib.aqlm_gemv_step_plan(_step_problems(9), nine, 1, 2, 8, 8, ctypes.addressof(buf), nbytes) == SHAPE
    one_level = (ctypes.c_int32 * 1)(1)
    for M, B in ((4, 8), (1, 8), (1, 16), (2, 12)):
        assert lib.aqlm_gemv_step_plan(probs, one_level, 1, M, B, 8, ctypes.addressof(buf), nbytes) == UNSUP
    # code rows that are not a multiple of 16 bytes, and x beyond the staging
    assert lib.aqlm_gemv_step_plan(_step_problems(1, d_in=1032), one_level, 1, 2, 8, 8, ctypes.addressof(buf),
                                   nbytes) == UNSUP
    assert lib.aqlm_gemv_step_plan(_step_problems(1, d_in=65536), one_level, 1, 2, 8, 8, ctypes.addressof(buf),
                                   nbytes) == UNSUP
    assert lib.aqlm_gemv_step_plan(_step_problems(1, d_out=0), one_level, 1, 2, 8, 8, ctypes.addressof(buf),
                                   nbytes) == SHAPE


def test_decode_step_launch_refusals(lib):
    """Checks that return before anything is launched (never a valid plan
    with fake pointers: that one would launch)."""
    nbytes = lib.aqlm_gemv_step_plan_bytes(1)
    buf = ctypes.create_string_buffer(nbytes)
    one_level = (ctypes.c_int32 * 1)(1)
    assert lib.aqlm_gemv_step_plan(_step_problems(1), one_level, 1, 2, 8, 8, ctypes.addressof(buf), nbytes) == OK
    assert lib.aqlm_gemv_step(None, P, P, 0, None) == NULL
    assert lib.aqlm_gemv_step(ctypes.addressof(buf), None, P, 0, None) == NULL
    assert lib.aqlm_gemv_step(ctypes.addressof(buf), P, None, 0, None) == NULL
    assert lib.aqlm_gemv_step(ctypes.addressof(buf), P + 8, P, 0, None) == ALIGN
    assert lib.aqlm_gemv_step(ctypes.addressof(buf), P, P + 4, 0, None) == ALIGN
    junk = ctypes.create_string_buffer(nbytes)
    assert lib.aqlm_gemv_step(ctypes.addressof(junk), P, P, 0, None) == SHAPE
    assert lib.aqlm_gemv_step_status(None, None) == NULL
    assert lib.aqlm_gemv_step_status(P + 4, None) == ALIGN


def test_large_groups_accepted_only_where_supported(lib):
    """g = 16, 32, 64 with 8-bit codes and up to 16 codebooks pass the checks
    of the entry points that take them (the calls then stop at the fake
    pointers' alignment); other shapes and entry points refuse them."""
    for M, g in ((4, 16), (8, 32), (15, 64), (16, 64), (1, 16)):
        assert deq(lib, M=M, g=g, d_in=128, w=P + 2) == ALIGN
        assert gemv(lib, M=M, g=g, d_in=128, y=P + 2) == ALIGN
        assert gemm(lib, M=M, g=g, d_in=128, y=P + 2) == ALIGN
        assert gemm_ws(lib, M=M, g=g, d_in=128, y=P + 2) == ALIGN
    for M, B, g in ((17, 8, 16), (4, 12, 16), (2, 16, 32), (4, 8, 128), (4, 8, 24), (0, 8, 16)):
        assert gemv(lib, M=M, B=B, g=g, d_in=384) == UNSUP, (M, B, g)
    assert gemv(lib, M=4, g=16, d_in=24) == SHAPE
    assert lib.aqlm_backward(P, P, P, 64, 64, 4, 8, 16, 4, P, P, P, P, None) == UNSUP
    assert lib.aqlm_beam_search(P, P, P, P, P, 8, 64, 4, 8, 16, 2, 1, P, None) == UNSUP
    Prob = _lib.GemvProblem
    arr = (Prob * 1)(Prob(P, P, P, P, P, 64, 64))
    assert lib.aqlm_gemv_grouped_path(arr, 1, 4, 8, 16, _lib.PATH_TABLE, None) == UNSUP
    nbytes = lib.aqlm_gemv_step_plan_bytes(1)
    buf = ctypes.create_string_buffer(nbytes)
    one = (ctypes.c_int32 * 1)(1)
    assert lib.aqlm_gemv_step_plan(arr, one, 1, 4, 8, 16, ctypes.addressof(buf), nbytes) == UNSUP


def tiled_bytes_by_definition(d_out, d_in, M):
    """Tiles of 16 rows x 64 code bytes, 1 KiB each, rows and row bytes
    rounded up to whole tiles."""
    row_bytes = d_in // 8 * M
    return -(-d_out // 16) * -(-row_bytes // 64) * 1024


def test_tiled_codes_validation(lib):
    """Tiled 8-bit codes: the size query, and bad arguments refused before
    anything is launched (fake pointers)."""
    for d_out, d_in, M in ((64, 256, 2), (37, 200, 2), (8192, 28672, 2), (1, 8, 1), (100, 520, 4)):
        assert lib.aqlm_tiled_codes_bytes(d_out, d_in, M, 8, 8) == tiled_bytes_by_definition(d_out, d_in, M)
    assert lib.aqlm_tiled_codes_bytes(64, 256, 3, 8, 8) == 0        # M = 3: no matrix-core kernel
    assert lib.aqlm_tiled_codes_bytes(64, 256, 1, 16, 8) == 0       # 16-bit codes
    assert lib.aqlm_tiled_codes_bytes(64, 256, 2, 8, 16) == 0       # groups of 16
    assert lib.aqlm_tiled_codes_bytes(0, 256, 2, 8, 8) == 0
    assert lib.aqlm_tiled_codes_bytes(64, 252, 2, 8, 8) == 0
    assert lib.aqlm_tiled_codes_bytes(1 << 20, 1 << 15, 4, 8, 8) == 0  # 2^31 bytes or more
    need = tiled_bytes_by_definition(64, 256, 2)
    assert lib.aqlm_tile_codes(None, 64, 256, 2, 8, 8, P, need, None) == NULL
    assert lib.aqlm_tile_codes(P, 64, 256, 2, 8, 8, None, need, None) == NULL
    assert lib.aqlm_tile_codes(P, 64, 256, 2, 8, 8, P, need - 1, None) == WORKSPACE
    assert lib.aqlm_tile_codes(P, 64, 256, 2, 8, 8, P + 8, need, None) == ALIGN
    assert lib.aqlm_tile_codes(P, 64, 256, 2, 16, 8, P, need, None) == UNSUP
    assert lib.aqlm_tile_codes(P, 64, 250, 2, 8, 8, P, need, None) == SHAPE
    Prob = _lib.GemvProblem
    good = Prob(P, P, P, P, P, 64, 256)
    arr = (Prob * 9)(*([good] * 9))
    assert lib.aqlm_gemv_grouped_tiled(None, 1, 2, 8, 8, None) == NULL
    assert lib.aqlm_gemv_grouped_tiled(arr, 0, 2, 8, 8, None) == SHAPE
    assert lib.aqlm_gemv_grouped_tiled(arr, 9, 2, 8, 8, None) == SHAPE
    assert lib.aqlm_gemv_grouped_tiled(arr, 2, 3, 8, 8, None) == UNSUP
    assert lib.aqlm_gemv_grouped_tiled(arr, 2, 1, 16, 8, None) == UNSUP
    bad = (Prob * 2)(good, Prob(P, P, P, P, P, 64, 60))
    assert lib.aqlm_gemv_grouped_tiled(bad, 2, 2, 8, 8, None) == SHAPE
    bad = (Prob * 2)(good, Prob(P + 8, P, P, P, P, 64, 256))
    assert lib.aqlm_gemv_grouped_tiled(bad, 2, 2, 8, 8, None) == ALIGN
    bad = (Prob * 2)(good, Prob(P, P, P, P, None, 64, 256))
    assert lib.aqlm_gemv_grouped_tiled(bad, 2, 2, 8, 8, None) == NULL


def test_tiled_grouped_validation_order(lib):
    """aqlm_gemv_grouped_tiled reports what aqlm_gemv_grouped reports first
    (a NULL pointer before an unsupported format)."""
    Prob = _lib.GemvProblem
    arr = (Prob * 1)(Prob(None, P, P, P, P, 64, 256))
    assert lib.aqlm_gemv_grouped(arr, 1, 1, 16, 8, None) == NULL
    assert lib.aqlm_gemv_grouped_tiled(arr, 1, 1, 16, 8, None) == NULL
    arr = (Prob * 1)(Prob(P, P, P, P, P, 64, 60))
    assert lib.aqlm_gemv_grouped_tiled(arr, 1, 3, 8, 8, None) == SHAPE


def test_tiled_small_batch_validation(lib):
    """aqlm_gemm_small_batch_tiled: aqlm_gemm_small_batch's checks first, then
    what the tiled product takes (1..64 rows; more than one row needs M of 2
    or 4), all before anything is launched (fake pointers: every call here
    must be refused)."""
    def call(codes=P, d_out=64, d_in=256, M=2, B=8, n=4, x=P, y=P):
        return lib.aqlm_gemm_small_batch_tiled(codes, P, P, d_out, d_in, M, B, 8, n, x, y, None)
    assert call(codes=None) == NULL
    assert call(x=None) == NULL
    assert call(n=0) == SHAPE
    assert call(d_in=250) == SHAPE
    assert call(x=P + 8) == ALIGN
    assert call(n=65) == UNSUP
    assert call(M=1, n=2) == UNSUP
    assert call(M=1, n=17) == UNSUP
    assert call(M=1, B=16) == UNSUP
    assert call(M=3) == UNSUP
