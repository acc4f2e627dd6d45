"""Parity of the matrix-vector product over chunk-sorted codes
(aqlm_gemv_sorted) with the CPU oracle, on the original row-major codes.

The sorted form is built by the library's host sorter (its layout is checked
in test_sorted_codes.py); the product must meet the same bar as aqlm_gemv:
relative L2 error 2e-3 and the elementwise bound of its fp32 arithmetic.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2401_06118_amd import synth
from paper_2401_06118_amd import format as aqfmt

from helpers import abs_codeword_sums, elementwise_bound, fp16_to_np, rel_l2, to_device

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


def check(lay, y, rows=None):
    """y: [d_out] fp16 numpy; rows: sampled rows (all when None)."""
    if rows is None:
        w = oracle.dequantize(lay.codes, lay.codebooks, lay.scales)
        got = y[None, :]
    else:
        w = oracle.dequantize_rows(lay.codes, lay.codebooks, lay.scales, rows)
        got = y[None, rows]
    ref = oracle.matmul_f16(w, lay.x)
    assert np.all(np.isfinite(got.astype(np.float64)))
    assert rel_l2(got, ref) <= TOL, rel_l2(got, ref)
    err = np.abs(got.astype(np.float64) - ref)
    bound = elementwise_bound(w, lay.x, ref, abs_codeword_sums(lay, rows))
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert np.all(err <= bound), ("elementwise", worst, err[worst], bound[worst])


FORMATS = [(1, 16), (1, 15), (2, 16), (2, 15)]


@pytest.mark.parametrize("M,B", FORMATS)
@pytest.mark.parametrize("d_out,d_in", [(4096, 4096), (11008, 4096), (4096, 11008), (1000, 4104), (37, 8),
                                        (40, 520), (513, 16384)])
def test_gemv_sorted_matches_oracle(M, B, d_out, d_in):
    """The 7B layer shapes, ragged row blocks (d_out not a multiple of 16),
    a single group per row, and x staged on chip (d_in up to 16376) or read
    through the cache (16384)."""
    print(f"[sorted gemv] {M}x{B} {d_out}x{d_in}", flush=True)
    lay = synth.layer(30_000 + 11 * B + 5 * M + d_out + d_in, d_out, d_in, M, B)
    codes, cb, sc, x = to_device(lay)
    sc_obj = aq().SortedCodes(codes, cb, sc)
    y = sc_obj.gemv(x[0])
    torch.cuda.synchronize()
    check(lay, fp16_to_np(y))


@pytest.mark.parametrize("d_out,d_in", [(28672, 8192), (8192, 28672)])
def test_gemv_sorted_70b_shapes_sampled_rows(d_out, d_in):
    """Llama-2-70B gate/up and down shapes with one codebook of 2^16: many
    blocks per row range, and an x too large to stage (read through the
    cache); rows sampled for the oracle."""
    print(f"[sorted gemv 70b] {d_out}x{d_in}", flush=True)
    lay = synth.layer(31_000 + d_out, d_out, d_in, 1, 16)
    codes, cb, sc, x = to_device(lay)
    y = aq().SortedCodes(codes, cb, sc).gemv(x[0])
    torch.cuda.synchronize()
    rows = np.random.default_rng(d_out).choice(d_out, size=96, replace=False)
    rows = np.sort(np.concatenate([rows, [0, 15, 16, d_out - 1]]))
    check(lay, fp16_to_np(y), rows)


def test_gemv_sorted_packed_input_same_result():
    """Sorting bit-packed 15-bit codes gives the same sorted form, hence the
    same product bit for bit."""
    lay = synth.layer(31_500, 1024, 4104, 1, 15)
    codes, cb, sc, x = to_device(lay)
    words = torch.from_numpy(np.ascontiguousarray(aqfmt.pack_codes(lay.codes, 15).view(np.int32))).cuda()
    y1 = aq().SortedCodes(codes, cb, sc).gemv(x[0])
    y2 = aq().SortedCodes(words, cb, sc, d_in=4104).gemv(x[0])
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    check(lay, fp16_to_np(y1))


def test_gemv_sorted_deterministic_and_workspace_reuse():
    """Repeated calls on one workspace give identical bits (each launch adds
    16 to the counters of its row ranges and tags its partial sums with the
    count), also interleaved with calls for a smaller layer of another format
    on the same workspace."""
    big = synth.layer(31_600, 4096, 4096, 1, 16)
    small = synth.layer(31_601, 300, 2048, 2, 16)  # 16 chunk classes
    codes_b, cb_b, sc_b, xb = to_device(big)
    s_big = aq().SortedCodes(codes_b, cb_b, sc_b)
    codes_s, cb_s, sc_s, xs = to_device(small)
    s_small = aq().SortedCodes(codes_s, cb_s, sc_s)
    s_small.workspace = s_big.workspace  # one workspace for both layers
    ys = []
    for k in range(100):
        ys.append(s_big.gemv(xb[0]).clone())
        if k % 10 == 0:
            ysm = s_small.gemv(xs[0])
    torch.cuda.synchronize()
    assert all(torch.equal(ys[0].view(torch.int16), y.view(torch.int16)) for y in ys[1:])
    check(big, fp16_to_np(ys[0]))
    check(small, fp16_to_np(ysm))
    counters = s_big.workspace[:4096].view(torch.int32)
    assert bool(torch.all(counters % 16 == 0)) and int(counters.max()) > 0


def test_gemv_sorted_zero_scales_and_cancelling_codewords():
    """Zero scales give zeros; codewords that cancel across the two codebooks
    stay within the bound of fp32 accumulation."""
    lay = synth.layer(31_700, 512, 4096, 2, 16)
    rng = np.random.default_rng(5)
    cbk = lay.codebooks.copy()
    big = (rng.standard_normal((1 << 16, 8)) * 64).astype(np.float16)
    cbk[0] = big
    cbk[1] = -big  # C_1[e] = -C_0[e]
    lay = dataclasses.replace(lay, codebooks=cbk)
    codes = lay.codes.copy()
    codes[:, :, 1] = codes[:, :, 0]  # every group adds C_0[e] + C_1[e] = 0 ...
    codes[::3, ::5, 1] ^= 1          # ... except where the second code differs
    lay = dataclasses.replace(lay, codes=codes)
    c, cb, sc, x = to_device(lay)
    y = aq().SortedCodes(c, cb, sc).gemv(x[0])
    zero = dataclasses.replace(lay, scales=np.zeros_like(lay.scales))
    c0, cb0, sc0, x0 = to_device(zero)
    y0 = aq().SortedCodes(c0, cb0, sc0).gemv(x0[0])
    torch.cuda.synchronize()
    check(lay, fp16_to_np(y))
    assert bool(torch.all(y0 == 0))


def test_gemv_sorted_agrees_with_gemv():
    """Same layer through aqlm_gemv and aqlm_gemv_sorted: both within the
    bound, and close to each other."""
    lay = synth.layer(31_800, 11008, 4096, 1, 16)
    codes, cb, sc, x = to_device(lay)
    y1 = aq().gemv(codes, cb, sc, x[0])
    y2 = aq().SortedCodes(codes, cb, sc).gemv(x[0])
    torch.cuda.synchronize()
    a, b = fp16_to_np(y1).astype(np.float64), fp16_to_np(y2).astype(np.float64)
    assert rel_l2(a, b) <= 1e-3
    check(lay, fp16_to_np(y2))


def test_gemv_sorted_argument_errors_touch_nothing():
    lay = synth.layer(31_900, 256, 1024, 1, 16)
    codes, cb, sc, x = to_device(lay)
    s = aq().SortedCodes(codes, cb, sc)
    out = torch.full((256,), 7.0, dtype=torch.float16, device="cuda")
    with pytest.raises(aq().AqlmError):
        import paper_2401_06118_amd._lib as L
        st = L.load().aqlm_gemv_sorted(s.entries.data_ptr(), s.entries.numel(), s.index.data_ptr(), None, cb.data_ptr(),
                                       sc.data_ptr(), 256, 1024, 1, 16, 8, x.data_ptr(), out.data_ptr(),
                                       s.workspace.data_ptr(), s.workspace.numel() - 1, None)
        aq()._check(st, "aqlm_gemv_sorted")
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)


@pytest.mark.parametrize("M,B", [(1, 16), (2, 15)])
def test_gemv_sorted_grouped_matches_oracle(M, B):
    """q, k, v-shaped problems sharing x, and gate/up-shaped ones, each in one
    launch; a ragged problem in the middle."""
    print(f"[sorted grouped] {M}x{B}", flush=True)
    for shapes in ([(4096, 4096), (1024, 4096), (1024, 4096)], [(11008, 4096), (37, 520), (11008, 4096)]):
        lays = [synth.layer(32_000 + 17 * i + B + M, o, i_, M, B) for i, (o, i_) in enumerate(shapes)]
        probs, ys = [], []
        for lay in lays:
            codes, cb, sc, x = to_device(lay)
            y = torch.empty(lay.codes.shape[0], dtype=torch.float16, device="cuda")
            probs.append((aq().SortedCodes(codes, cb, sc), x[0], y))
            ys.append(y)
        aq().gemv_sorted_grouped(probs)
        torch.cuda.synchronize()
        for lay, y in zip(lays, ys):
            check(lay, fp16_to_np(y))
        # the same products one by one agree closely
        for (s, x, y) in probs:
            y1 = s.gemv(x)
            torch.cuda.synchronize()
            assert rel_l2(fp16_to_np(y1).astype(np.float64), fp16_to_np(y).astype(np.float64)) <= 1e-3


def test_gemv_sorted_grouped_deterministic():
    lays = [synth.layer(32_100 + i, 4096, 4096, 1, 16) for i in range(3)]
    probs = []
    for lay in lays:
        codes, cb, sc, x = to_device(lay)
        probs.append((aq().SortedCodes(codes, cb, sc), x[0], torch.empty(4096, dtype=torch.float16, device="cuda")))
    outs = []
    for _ in range(20):
        aq().gemv_sorted_grouped(probs)
        outs.append(torch.cat([p[2] for p in probs]).clone())
    torch.cuda.synchronize()
    assert all(torch.equal(outs[0].view(torch.int16), o.view(torch.int16)) for o in outs[1:])


def test_gemv_sorted_without_host_index_same_bits():
    """Without the host copy of the index the workgroups read their first
    steps from the device index: same results bit for bit."""
    import paper_2401_06118_amd._lib as L
    for (d_out, d_in) in [(4096, 4096), (1000, 4104), (8192, 28672)]:
        lay = synth.layer(32_200 + d_out, d_out, d_in, 1, 16)
        codes, cb, sc, x = to_device(lay)
        s = aq().SortedCodes(codes, cb, sc)
        y1 = s.gemv(x[0])
        y2 = torch.empty_like(y1)
        st = L.load().aqlm_gemv_sorted(s.entries.data_ptr(), s.entries.numel(), s.index.data_ptr(), None,
                                       cb.data_ptr(), sc.data_ptr(), d_out, d_in, 1, 16, 8, x.data_ptr(),
                                       y2.data_ptr(), s.workspace.data_ptr(), s.workspace.numel(), None)
        assert st == 0
        torch.cuda.synchronize()
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("d_out,d_in", [(1, 2048), (16, 8), (210_000, 64)])
def test_gemv_sorted_extreme_shapes(d_out, d_in):
    """One row; one block of one group; and a layer tall enough to need more
    row ranges than one workgroup round holds (13125 blocks: 33 ranges of at
    most 400 blocks, 264 workgroups on 256 CUs, so the workgroups' step
    ranges come from the device index and the summing workgroups poll
    partners that run in the same round or an earlier one)."""
    print(f"[sorted extreme] {d_out}x{d_in}", flush=True)
    lay = synth.layer(33_000 + d_out + d_in, d_out, d_in, 1, 16)
    codes, cb, sc, x = to_device(lay)
    y = aq().SortedCodes(codes, cb, sc).gemv(x[0])
    torch.cuda.synchronize()
    if d_out <= 4096:
        check(lay, fp16_to_np(y))
    else:
        rows = np.sort(np.random.default_rng(d_out).choice(d_out, size=200, replace=False))
        rows = np.unique(np.concatenate([rows, [0, 6399, 6400, d_out - 1]]))
        check(lay, fp16_to_np(y), rows)
