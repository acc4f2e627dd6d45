"""Host-side checks of the chunk-sorted code form (aqlm_sort_codes): the
layout include/aqlm.h defines, rebuilt here from the row-major codes with
numpy, and the argument checks of the three sorted-code entry points.  The
sorter runs on the host, so no GPU is needed."""
import ctypes
import os

import numpy as np
import pytest

from paper_2401_06118_amd import _lib
from paper_2401_06118_amd import format as aqfmt

OK, NULL, SHAPE, UNSUP, ALIGN, WORKSPACE = 0, 1, 2, 3, 4, 6
PAD = 0xFFFFE000
P = 0x10000  # fake device address, never dereferenced on error paths


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.skip("library not built (run python -m paper_2401_06118_amd.build)")
    return _lib.load()


def sort(lib, codes, d_out, d_in, M, B):
    """(entries uint32, index uint32) from the library's host sorter."""
    src = np.ascontiguousarray(codes)
    ew, iw = ctypes.c_int64(0), ctypes.c_int64(0)
    st = lib.aqlm_sort_codes_size(src.ctypes.data, d_out, d_in, M, B, 8, ctypes.byref(ew), ctypes.byref(iw))
    assert st == OK, st
    entries = np.empty(ew.value, dtype=np.uint32)
    index = np.empty(iw.value, dtype=np.uint32)
    st = lib.aqlm_sort_codes(src.ctypes.data, d_out, d_in, M, B, 8, entries.ctypes.data, ew.value,
                             index.ctypes.data, iw.value)
    assert st == OK, st
    return entries, index


def expected_layout(codes, B):
    """The sorted form written out from its definition: per 16-row block and
    chunk class, the rows' codes of that class in ascending group order, four
    lanes per row per step of 64 entries."""
    d_out, G, M = codes.shape
    K = M << (B - 13)
    nb = (d_out + 15) // 16
    cls = (np.arange(M)[None, None, :] << (B - 13)) + (codes.astype(np.int64) >> 13)
    steps = np.zeros((K, nb), dtype=np.int64)
    lists = {}
    for b in range(nb):
        rows = range(16 * b, min(16 * b + 16, d_out))
        for c in range(K):
            per_row = []
            for i in rows:
                jj, mm = np.nonzero(cls[i] == c)  # row-major over (j, m): ascending j
                per_row.append([(int(codes[i, j, m]) & 8191) | (int(j) << 14) for j, m in zip(jj, mm)])
            lists[c, b] = per_row
            steps[c, b] = (max(len(r) for r in per_row) + 3) // 4
    index = np.concatenate([[0], np.cumsum(steps.reshape(-1))]).astype(np.uint32)
    entries = np.full(int(index[-1]) * 64, PAD, dtype=np.uint32)
    for (c, b), per_row in lists.items():
        base = int(index[c * nb + b])
        for i, row in enumerate(per_row):
            for k, e in enumerate(row):
                entries[64 * (base + k // 4) + 16 * (k % 4) + i] = e
    return entries, index


CASES = [
    # (d_out, d_in, M, B)
    (16, 256, 1, 16), (40, 520, 1, 16), (7, 8, 1, 16), (33, 1024, 1, 15),
    (48, 512, 2, 16), (21, 136, 2, 15), (1, 2048, 1, 16),
]


@pytest.mark.parametrize("d_out,d_in,M,B", CASES)
def test_sorted_layout_matches_definition(lib, d_out, d_in, M, B):
    rng = np.random.default_rng(1000 + d_out + d_in + M + B)
    codes = rng.integers(0, 1 << B, size=(d_out, d_in // 8, M), dtype=np.uint16)
    got_e, got_i = sort(lib, codes, d_out, d_in, M, B)
    want_e, want_i = expected_layout(codes, B)
    np.testing.assert_array_equal(got_i, want_i)
    np.testing.assert_array_equal(got_e, want_e)


def test_sorted_layout_high_bits_and_skewed_classes(lib):
    """Bits above B are ignored (as in every entry point), and codes that all
    fall in one chunk give empty lists for the other classes."""
    d_out, d_in, M, B = 32, 512, 1, 15
    rng = np.random.default_rng(7)
    codes = rng.integers(0, 8192, size=(d_out, d_in // 8, M), dtype=np.uint16) | np.uint16(0x8000)
    got_e, got_i = sort(lib, codes, d_out, d_in, M, B)
    want_e, want_i = expected_layout(codes & np.uint16(0x7FFF), B)
    np.testing.assert_array_equal(got_i, want_i)
    np.testing.assert_array_equal(got_e, want_e)
    nb = 2
    steps = np.diff(got_i.astype(np.int64)).reshape(4, nb)
    assert np.all(steps[1:] == 0) and np.all(steps[0] == (d_in // 8) // 4)


@pytest.mark.parametrize("M,B", [(1, 15), (2, 15)])
def test_sorted_form_of_packed_codes_is_the_same(lib, M, B):
    d_out, d_in = 40, 1032
    rng = np.random.default_rng(11 + M)
    codes = rng.integers(0, 1 << B, size=(d_out, d_in // 8, M), dtype=np.uint16)
    words = aqfmt.pack_codes(codes, B)
    e1, i1 = sort(lib, codes, d_out, d_in, M, B)
    e2, i2 = sort(lib, words, d_out, d_in, M, B | _lib.PACKED)
    np.testing.assert_array_equal(i1, i2)
    np.testing.assert_array_equal(e1, e2)


def test_every_code_appears_once(lib):
    """A 4096 x 4096 1x16 layer: decoding the entries back gives every
    (row, group) code exactly once."""
    d_out, d_in, M, B = 4096, 4096, 1, 16
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 1 << B, size=(d_out, d_in // 8, M), dtype=np.uint16)
    entries, index = sort(lib, codes, d_out, d_in, M, B)
    nb, K = d_out // 16, 8
    back = np.full((d_out, d_in // 8), -1, dtype=np.int64)
    for c in range(K):
        for b in range(nb):
            s0, s1 = int(index[c * nb + b]), int(index[c * nb + b + 1])
            blk = entries[64 * s0:64 * s1].reshape(-1, 64)
            for lane_row in range(16):
                e = blk[:, lane_row::16].reshape(-1)
                e = e[e != PAD]
                j = (e >> 14).astype(np.int64)
                assert np.all(back[16 * b + lane_row, j] == -1)
                back[16 * b + lane_row, j] = (c << 13) | (e & 8191)
    np.testing.assert_array_equal(back, codes[:, :, 0].astype(np.int64))
    # pads: about a quarter of the entries at 512 codes per row
    assert 0.15 < np.mean(entries == PAD) < 0.3


def test_sort_refusals(lib):
    codes = np.zeros((16, 8, 1), dtype=np.uint16)
    ew, iw = ctypes.c_int64(0), ctypes.c_int64(0)
    size = lambda d_out, d_in, M, B, g=8, src=codes.ctypes.data: lib.aqlm_sort_codes_size(  # noqa: E731
        src, d_out, d_in, M, B, g, ctypes.byref(ew), ctypes.byref(iw))
    assert size(16, 64, 1, 16) == OK and ew.value > 0 and iw.value == 8 + 1
    assert size(16, 64, 1, 16, src=None) == NULL
    assert lib.aqlm_sort_codes_size(codes.ctypes.data, 16, 64, 1, 16, 8, None, ctypes.byref(iw)) == NULL
    for M, B in [(2, 8), (1, 12), (2, 12), (3, 16), (1, 14)]:
        assert size(16, 64, M, B) == UNSUP, (M, B)
    assert size(16, 64, 1, 16 | _lib.PACKED) == UNSUP  # 16-bit codes have no packed form
    assert size(16, 64, 1, 16, g=16) == UNSUP
    assert size(0, 64, 1, 16) == SHAPE and size(16, 60, 1, 16) == SHAPE
    e = np.empty(ew.value, dtype=np.uint32)
    i = np.empty(iw.value, dtype=np.uint32)
    sort_ = lib.aqlm_sort_codes
    assert sort_(codes.ctypes.data, 16, 64, 1, 16, 8, e.ctypes.data, ew.value - 1, i.ctypes.data, iw.value) == \
        WORKSPACE
    assert sort_(codes.ctypes.data, 16, 64, 1, 16, 8, e.ctypes.data, ew.value, i.ctypes.data, iw.value - 1) == \
        WORKSPACE
    assert sort_(codes.ctypes.data, 16, 64, 1, 16, 8, None, ew.value, i.ctypes.data, iw.value) == NULL


def test_gemv_sorted_refuses_before_launch(lib):
    """Every refusal comes from host checks (fake device pointers)."""
    ws = lib.aqlm_gemv_sorted_workspace_bytes(4096, 1, 16)
    assert ws == 4096 + 8 * 4096 * 8
    assert lib.aqlm_gemv_sorted_workspace_bytes(4096, 2, 16) == 4096 + 16 * 4096 * 8
    assert lib.aqlm_gemv_sorted_workspace_bytes(4096, 2, 8) == 0
    assert lib.aqlm_gemv_sorted_workspace_bytes(0, 1, 16) == 0

    def call(entries=P, ew=64 * 100, index=P, cb=P, sc=P, d_out=4096, d_in=4096, M=1, B=16, g=8, x=P, y=P,
             w=P, wb=ws):
        return lib.aqlm_gemv_sorted(entries, ew, index, None, cb, sc, d_out, d_in, M, B, g, x, y, w, wb, None)

    for kw in ("entries", "index", "cb", "sc", "x", "y", "w"):
        assert call(**{kw: None}) == NULL, kw
    assert call(M=2, B=8) == UNSUP and call(B=12, M=2) == UNSUP and call(g=16) == UNSUP
    assert call(B=16 | _lib.PACKED) == UNSUP
    assert call(d_in=4100) == SHAPE and call(d_out=0) == SHAPE
    assert call(ew=0) == SHAPE and call(ew=100) == SHAPE
    assert call(d_out=6553601, wb=lib.aqlm_gemv_sorted_workspace_bytes(6553601, 1, 16)) == SHAPE
    assert call(wb=ws - 1) == WORKSPACE
    assert call(entries=P + 2) == ALIGN and call(x=P + 8) == ALIGN and call(w=P + 4) == ALIGN
    assert call(cb=P + 8) == ALIGN and call(y=P + 1) == ALIGN


def test_gemv_sorted_grouped_refuses_before_launch(lib):
    """Grouped calls validate every problem and the summed workspace first."""
    def prob(d_out=4096, d_in=4096, ew=64 * 100, entries=P, x=P):
        return _lib.SortedProblem(entries, ew, P, None, P, P, x, P, d_out, d_in)

    def call(probs, M=1, B=16, wb=None, ws=P):
        arr = (_lib.SortedProblem * max(len(probs), 1))(*probs)
        rows = sum(p.d_out for p in probs)
        if wb is None:
            wb = lib.aqlm_gemv_sorted_workspace_bytes(max(rows, 1), M, B)
        return lib.aqlm_gemv_sorted_grouped(arr, len(probs), M, B, 8, ws, wb, None)

    assert call([prob(), prob()], wb=lib.aqlm_gemv_sorted_workspace_bytes(4096, 1, 16)) == WORKSPACE
    assert call([prob(), prob(entries=None)]) == NULL
    assert call([prob(), prob(d_in=4100)]) == SHAPE
    assert call([prob(), prob(x=P + 2)]) == ALIGN
    assert call([prob()] * 9) == SHAPE
    assert call([prob()], ws=None) == NULL
    assert call([prob()], M=2, B=8) == UNSUP
    # at most 1024 row ranges of 400 blocks per launch
    assert call([prob(d_out=4_000_000), prob(d_out=4_000_000)]) == SHAPE
