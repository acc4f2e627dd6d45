"""MI355X-native AQLM inference path.

AQLM (Additive Quantization of Language Models) stores a weight matrix as
codes into M learned codebooks plus one scale per output unit (paper: Sec. 3,
Eq. 2 and Fig. 3).  This package exposes the three operations of the C ABI in
``include/aqlm.h`` on torch tensors that live on the GPU:

- :func:`dequantize` - rebuild the fp16 weight matrix, bit-exact;
- :func:`gemv` - the token-generation matrix-vector product (Sec. 4.3);
- :func:`gemv_grouped` - several independent matrix-vector products in one launch;
- :func:`gemm_small_batch` - the same product for n activation rows;
- :func:`gemm` - that product with a workspace: for many rows the weights are
  dequantized once, then a dense fp16 matrix-core product reads them;
- :func:`backward` - gradients of the codebooks and scales through Eq. 2;
- :func:`beam_search` - Phase 1 of the quantizer: beam search over the codes;
- :class:`DecodeStep` - the products of a whole decode step (levels of
  grouped 2x8 products, each level free to read what earlier ones wrote) as
  one persistent launch;
- :class:`SortedCodes` - a chunk-sorted copy of the codes of the large-codebook
  formats (1x15, 1x16, 2x15, 2x16) whose matrix-vector product serves every
  code from a codebook chunk held on chip.

Every computation runs in the hand-written HIP kernels of
``libaqlm_mi355x.so``; this module only marshals arguments.

Tensor formats: ``codes`` uint8 [d_out, d_in/8, M] (B = 8) or uint16/int16
[d_out, d_in/8, M] (B = 12, 15, 16); ``codebooks`` fp16 [M, 2^B, 8]; ``scales``
fp16 [d_out] (a trailing singleton dimension is accepted); activations fp16.
:func:`dequantize`, :func:`gemv` and :func:`gemv_grouped` also take bit-packed
codes (B = 12 or 15): int32 [d_out, row words], each row a little-endian bit
string of its d_in/8 * M codes (code (j, m) at bits (j*M + m)*B ..), zero-padded
to whole 32-bit words (``format.pack_codes`` writes it).
"""
from __future__ import annotations

import ctypes

import torch

from . import _lib
from ._lib import AqlmError, status_string  # noqa: F401

__all__ = ["dequantize", "gemv", "gemv_grouped", "gemm_small_batch", "gemm_workspace_bytes", "gemm", "backward",
           "beam_search", "DecodeStep", "SortedCodes", "gemv_sorted_grouped",
           "AqlmError",
           "status_string", "layer_args", "packed_layer_args"]


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def layer_args(codes: torch.Tensor, codebooks: torch.Tensor, scales: torch.Tensor):
    """Validate tensor metadata and return (d_out, d_in, M, B, g)."""
    for name, t in (("codes", codes), ("codebooks", codebooks), ("scales", scales)):
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if codebooks.dtype != torch.float16 or codebooks.dim() != 3:
        raise ValueError("codebooks must be fp16 [M, 2^B, g]")
    M, entries, g = codebooks.shape
    B = int(entries).bit_length() - 1
    if (1 << B) != entries:
        raise ValueError("codebook entry count must be a power of two")
    if codes.dim() != 3 or codes.shape[2] != M:
        raise ValueError("codes must be [d_out, d_in/g, M]")
    want = (torch.uint8,) if B <= 8 else (torch.uint16, torch.int16)
    if codes.dtype not in want:
        raise ValueError(f"codes for B={B} must be {want[0]}")
    if scales.dtype != torch.float16 or scales.numel() != codes.shape[0]:
        raise ValueError("scales must be fp16 with one value per output row")
    d_out, groups, _ = codes.shape
    return d_out, groups * g, M, B, g


def packed_layer_args(words: torch.Tensor, codebooks: torch.Tensor, scales: torch.Tensor, d_in: int):
    """Validate bit-packed codes (int32 [d_out, row words]) and return
    (d_out, d_in, M, B | PACKED, g) for the C ABI."""
    for name, t in (("codes", words), ("codebooks", codebooks), ("scales", scales)):
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if codebooks.dtype != torch.float16 or codebooks.dim() != 3:
        raise ValueError("codebooks must be fp16 [M, 2^B, g]")
    M, entries, g = codebooks.shape
    B = int(entries).bit_length() - 1
    if (1 << B) != entries:
        raise ValueError("codebook entry count must be a power of two")
    if words.dtype != torch.int32 or words.dim() != 2:
        raise ValueError("packed codes must be int32 [d_out, row words]")
    d_in = int(d_in)
    if d_in <= 0 or d_in % g != 0:
        raise ValueError(f"d_in must be a positive multiple of {g}")
    row_words = ((d_in // g) * M * B + 31) // 32
    if words.shape[1] != row_words:
        raise ValueError(f"packed codes of d_in={d_in}, M={M}, B={B} have {row_words} words per row")
    if scales.dtype != torch.float16 or scales.numel() != words.shape[0]:
        raise ValueError("scales must be fp16 with one value per output row")
    return words.shape[0], d_in, M, B | _lib.PACKED, g


def _args(codes, codebooks, scales, d_in):
    """layer_args, or packed_layer_args for 2-D (bit-packed) codes."""
    if codes.dim() == 2:
        if d_in is None:
            raise ValueError("bit-packed codes need d_in")
        return packed_layer_args(codes, codebooks, scales, d_in)
    return layer_args(codes, codebooks, scales)


def _out(out, shape, like: torch.Tensor) -> torch.Tensor:
    """A caller's output tensor, checked like the inputs (the C ABI cannot see
    sizes, so an undersized buffer would be written past its end), or a new
    one."""
    if out is None:
        return torch.empty(shape, dtype=torch.float16, device=like.device)
    if not isinstance(out, torch.Tensor) or out.dtype != torch.float16 or not out.is_cuda:
        raise ValueError("out must be an fp16 GPU tensor")
    if not out.is_contiguous():
        raise ValueError("out must be contiguous")
    if tuple(out.shape) != tuple(shape):
        raise ValueError(f"out must have shape {tuple(shape)}, got {tuple(out.shape)}")
    if out.device != like.device:
        raise ValueError("out must be on the same device as the layer")
    return out


def _check(st: int, what: str):
    if st != _lib.AQLM_OK:
        raise AqlmError(st, what)


def dequantize(codes, codebooks, scales, *, d_in=None, out=None, stream=None) -> torch.Tensor:
    """fp16 weight matrix [d_out, d_in]: w[i, 8j+k] = fp16(sum_m C_m[b_ijm][k] * s_i).
    ``d_in`` is needed (only) for bit-packed codes."""
    d_out, d_in, M, B, g = _args(codes, codebooks, scales, d_in)
    out = _out(out, (d_out, d_in), codes)
    st = _lib.load().aqlm_dequantize(codes.data_ptr(), codebooks.data_ptr(), scales.data_ptr(), d_out, d_in,
                                     M, B, g, out.data_ptr(), _stream_handle(stream))
    _check(st, "aqlm_dequantize")
    return out


def gemv(codes, codebooks, scales, x, *, out=None, stream=None) -> torch.Tensor:
    """y [d_out] = W x for one fp16 activation vector x [d_in]."""
    d_out, d_in, M, B, g = _args(codes, codebooks, scales, x.numel())
    if x.dtype != torch.float16 or x.numel() != d_in or not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous fp16 GPU tensor with d_in elements")
    out = _out(out, (d_out,), codes)
    st = _lib.load().aqlm_gemv(codes.data_ptr(), codebooks.data_ptr(), scales.data_ptr(), d_out, d_in, M, B, g,
                               x.data_ptr(), out.data_ptr(), _stream_handle(stream))
    _check(st, "aqlm_gemv")
    return out


def gemv_grouped(problems, *, path: str = "auto", stream=None):
    """Independent products [(codes, codebooks, scales, x, y), ...] sharing (M, B)
    in one launch; each y [d_out] is written in place.  Returns the y list.
    ``path``: "auto" (the library's choice), "gather" (codeword gathers) or
    "table" (per-group partial-product tables; 2x8, d_in % 256 == 0)."""
    paths = {"auto": _lib.PATH_AUTO, "gather": _lib.PATH_GATHER, "table": _lib.PATH_TABLE}
    if path not in paths:
        raise ValueError(f"path must be one of {sorted(paths)}")
    if not 1 <= len(problems) <= _lib.MAX_GROUPED:
        raise ValueError(f"1..{_lib.MAX_GROUPED} problems per grouped launch")
    arr = (_lib.GemvProblem * len(problems))()
    fmt = None
    for i, (codes, codebooks, scales, x, y) in enumerate(problems):
        d_out, d_in, M, B, g = _args(codes, codebooks, scales, x.numel())
        if fmt is None:
            fmt = (M, B, g)
        elif fmt != (M, B, g):
            raise ValueError("grouped problems must share (M, B, g)")
        if x.dtype != torch.float16 or x.numel() != d_in or not x.is_cuda or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 GPU tensor with d_in elements")
        if y.dtype != torch.float16 or y.numel() != d_out or not y.is_cuda or not y.is_contiguous():
            raise ValueError("y must be a contiguous fp16 GPU tensor with d_out elements")
        arr[i] = _lib.GemvProblem(codes.data_ptr(), codebooks.data_ptr(), scales.data_ptr(), x.data_ptr(),
                                  y.data_ptr(), d_out, d_in)
    st = _lib.load().aqlm_gemv_grouped_path(arr, len(problems), fmt[0], fmt[1], fmt[2], paths[path],
                                            _stream_handle(stream))
    _check(st, "aqlm_gemv_grouped_path")
    return [p[4] for p in problems]


class TiledCodes:
    """Tiled copy of a layer's 8-bit codes for the batch-1 product
    (``aqlm_tile_codes`` / ``aqlm_gemv_grouped_tiled``): the codes of every
    16 rows x 64-byte K-slice stored as one contiguous 1 KiB tile, written on
    the GPU once.  ``codes``: uint8 [d_out, d_in/8, M] as for :func:`gemv`
    (M of 1, 2 or 4, 2^8 codewords).  The products equal those over the
    row-major codes bit for bit."""

    def __init__(self, codes, codebooks, scales, *, stream=None):
        d_out, d_in, M, B, g = _args(codes, codebooks, scales, None)
        lib = _lib.load()
        need = int(lib.aqlm_tiled_codes_bytes(d_out, d_in, M, B, g))
        if need <= 0:
            raise ValueError("tiled codes take 8-bit codes with M in {1, 2, 4} and g = 8")
        self.codes = torch.empty(need, dtype=torch.uint8, device=codes.device)
        _check(lib.aqlm_tile_codes(codes.data_ptr(), d_out, d_in, M, B, g, self.codes.data_ptr(), need,
                                   _stream_handle(stream)), "aqlm_tile_codes")
        self.codebooks, self.scales = codebooks, scales
        self.d_out, self.d_in, self.M, self.B, self.g = d_out, d_in, M, B, g

    def gemm_small_batch(self, x, *, out=None, stream=None) -> torch.Tensor:
        """Y [n, d_out] = X W^T for fp16 activations X [n, d_in], 1 <= n <= 64
        (n > 1 needs M of 2 or 4): what :func:`gemm_small_batch` computes on
        the row-major codes, bit for bit."""
        if x.dtype != torch.float16 or x.dim() != 2 or x.shape[1] != self.d_in or not x.is_cuda \
                or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 GPU tensor [n, d_in]")
        n = x.shape[0]
        out = _out(out, (n, self.d_out), self.codes)
        st = _lib.load().aqlm_gemm_small_batch_tiled(self.codes.data_ptr(), self.codebooks.data_ptr(),
                                                     self.scales.data_ptr(), self.d_out, self.d_in, self.M, self.B,
                                                     self.g, n, x.data_ptr(), out.data_ptr(), _stream_handle(stream))
        _check(st, "aqlm_gemm_small_batch_tiled")
        return out


def gemv_tiled_grouped(problems, *, stream=None):
    """Independent products [(tiled, x, y), ...] (``TiledCodes`` sharing
    (M, B, g)) in one launch; each y [d_out] is written in place.  Returns
    the y list."""
    if not 1 <= len(problems) <= _lib.MAX_GROUPED:
        raise ValueError(f"1..{_lib.MAX_GROUPED} problems per grouped launch")
    arr = (_lib.GemvProblem * len(problems))()
    fmt = None
    for i, (t, x, y) in enumerate(problems):
        if fmt is None:
            fmt = (t.M, t.B, t.g)
        elif fmt != (t.M, t.B, t.g):
            raise ValueError("grouped problems must share (M, B, g)")
        if x.dtype != torch.float16 or x.numel() != t.d_in or not x.is_cuda or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 GPU tensor with d_in elements")
        if y.dtype != torch.float16 or y.numel() != t.d_out or not y.is_cuda or not y.is_contiguous():
            raise ValueError("y must be a contiguous fp16 GPU tensor with d_out elements")
        arr[i] = _lib.GemvProblem(t.codes.data_ptr(), t.codebooks.data_ptr(), t.scales.data_ptr(), x.data_ptr(),
                                  y.data_ptr(), t.d_out, t.d_in)
    st = _lib.load().aqlm_gemv_grouped_tiled(arr, len(problems), fmt[0], fmt[1], fmt[2], _stream_handle(stream))
    _check(st, "aqlm_gemv_grouped_tiled")
    return [p[2] for p in problems]


def gemm_small_batch(codes, codebooks, scales, x, *, out=None, stream=None) -> torch.Tensor:
    """Y [n, d_out] = X W^T for fp16 activations X [n, d_in]."""
    d_out, d_in, M, B, g = layer_args(codes, codebooks, scales)
    if x.dtype != torch.float16 or x.dim() != 2 or x.shape[1] != d_in or not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous fp16 GPU tensor [n, d_in]")
    n = x.shape[0]
    out = _out(out, (n, d_out), codes)
    st = _lib.load().aqlm_gemm_small_batch(codes.data_ptr(), codebooks.data_ptr(), scales.data_ptr(), d_out, d_in,
                                           M, B, g, n, x.data_ptr(), out.data_ptr(), _stream_handle(stream))
    _check(st, "aqlm_gemm_small_batch")
    return out


def gemm_workspace_bytes(codes, codebooks, scales, n: int) -> int:
    """Bytes of device workspace :func:`gemm` needs for n activation rows (0: none)."""
    d_out, d_in, M, B, g = layer_args(codes, codebooks, scales)
    return int(_lib.load().aqlm_gemm_workspace_bytes(d_out, d_in, M, B, g, int(n)))


def gemm(codes, codebooks, scales, x, *, workspace=None, out=None, stream=None) -> torch.Tensor:
    """Y [n, d_out] = X W^T like :func:`gemm_small_batch`, through ``aqlm_gemm``.
    ``workspace``: a GPU tensor of at least :func:`gemm_workspace_bytes` bytes;
    allocated here (by torch) when not given and needed."""
    d_out, d_in, M, B, g = layer_args(codes, codebooks, scales)
    if x.dtype != torch.float16 or x.dim() != 2 or x.shape[1] != d_in or not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous fp16 GPU tensor [n, d_in]")
    n = x.shape[0]
    need = int(_lib.load().aqlm_gemm_workspace_bytes(d_out, d_in, M, B, g, n))
    if workspace is None and need > 0:
        workspace = torch.empty((need,), dtype=torch.uint8, device=codes.device)
    if workspace is not None and (not workspace.is_cuda or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous GPU tensor")
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    out = _out(out, (n, d_out), codes)
    st = _lib.load().aqlm_gemm(codes.data_ptr(), codebooks.data_ptr(), scales.data_ptr(), d_out, d_in, M, B, g, n,
                               x.data_ptr(), out.data_ptr(), ws_ptr, ws_bytes, _stream_handle(stream))
    _check(st, "aqlm_gemm")
    return out


def backward(codes, codebooks, scales, x, dy, *, dcodebooks=None, dscales=None, stream=None):
    """Gradients through Eq. 2 for y = x W^T: accumulates dL/dC into
    ``dcodebooks`` (fp32 [M, 2^B, g]) and dL/ds into ``dscales`` (fp32 [d_out]),
    new zero tensors when not given; returns (dcodebooks, dscales).  x [n, d_in]
    and dy = dL/dy [n, d_out] are fp16."""
    d_out, d_in, M, B, g = layer_args(codes, codebooks, scales)
    for name, t, shape in (("x", x, (None, d_in)), ("dy", dy, (None, d_out))):
        if t.dtype != torch.float16 or t.dim() != 2 or t.shape[1] != shape[1] or not t.is_cuda \
                or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp16 GPU tensor [n, {shape[1]}]")
    n = x.shape[0]
    if dy.shape[0] != n:
        raise ValueError("x and dy must have the same number of rows")
    if dcodebooks is None:
        dcodebooks = torch.zeros(tuple(codebooks.shape), dtype=torch.float32, device=codes.device)
    if dscales is None:
        dscales = torch.zeros((d_out,), dtype=torch.float32, device=codes.device)
    for name, t, shape in (("dcodebooks", dcodebooks, tuple(codebooks.shape)), ("dscales", dscales, (d_out,))):
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp32 GPU tensor of shape {shape}")
    st = _lib.load().aqlm_backward(codes.data_ptr(), codebooks.data_ptr(), scales.data_ptr(), d_out, d_in, M, B, g,
                                   n, x.data_ptr(), dy.data_ptr(), dcodebooks.data_ptr(), dscales.data_ptr(),
                                   _stream_handle(stream))
    _check(st, "aqlm_backward")
    return dcodebooks, dscales


def beam_search(w, h, codes, codebooks, scales, *, beam: int, sweeps: int = 1, stream=None) -> torch.Tensor:
    """Phase-1 beam search over the codes of every row for the objective
    (w_i - what_i) H (w_i - what_i)^T, H = X X^T; ``codes`` (uint8 [d_out, d_in/8, M])
    is improved in place.  w: fp32 [d_out, d_in]; h: fp32 [d_in, d_in].
    Returns each row's final loss (fp32 [d_out])."""
    d_out, d_in, M, B, g = layer_args(codes, codebooks, scales)
    for name, t, shape in (("w", w, (d_out, d_in)), ("h", h, (d_in, d_in))):
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp32 GPU tensor of shape {shape}")
    loss = torch.empty((d_out,), dtype=torch.float32, device=codes.device)
    st = _lib.load().aqlm_beam_search(w.data_ptr(), h.data_ptr(), codes.data_ptr(), codebooks.data_ptr(),
                                      scales.data_ptr(), d_out, d_in, M, B, g, int(beam), int(sweeps),
                                      loss.data_ptr(), _stream_handle(stream))
    _check(st, "aqlm_beam_search")
    return loss


class DecodeStep:
    """A planned decode step: ``levels`` is a list of levels, each a list of
    (codes, codebooks, scales, x, y) 2x8 problems as for :func:`gemv_grouped`.
    Level l + 1 reads its x only after level l has written every y, so a
    level's x may be an earlier level's y.  The plan is built on the host,
    copied to the device once, and :meth:`run` launches the whole step as one
    persistent kernel.  The tensors must outlive the plan (it holds their
    device pointers; references are kept here)."""

    def __init__(self, levels, *, device=None):
        import ctypes
        if not levels:
            raise ValueError("a step needs at least one level")
        probs, sizes, keep = [], [], []
        fmt = None
        for lv in levels:
            if not 1 <= len(lv) <= _lib.MAX_GROUPED:
                raise ValueError(f"1..{_lib.MAX_GROUPED} problems per level")
            sizes.append(len(lv))
            for codes, codebooks, scales, x, y in lv:
                d_out, d_in, M, B, g = layer_args(codes, codebooks, scales)
                if fmt is None:
                    fmt = (M, B, g)
                elif fmt != (M, B, g):
                    raise ValueError("all problems of a step must share (M, B, g)")
                if x.dtype != torch.float16 or x.numel() != d_in or not x.is_cuda or not x.is_contiguous():
                    raise ValueError("x must be a contiguous fp16 GPU tensor with d_in elements")
                if y.dtype != torch.float16 or y.numel() != d_out or not y.is_cuda or not y.is_contiguous():
                    raise ValueError("y must be a contiguous fp16 GPU tensor with d_out elements")
                probs.append(_lib.GemvProblem(codes.data_ptr(), codebooks.data_ptr(), scales.data_ptr(),
                                              x.data_ptr(), y.data_ptr(), d_out, d_in))
                keep.append((codes, codebooks, scales, x, y))
        lib = _lib.load()
        n = len(sizes)
        nbytes = int(lib.aqlm_gemv_step_plan_bytes(n))
        if nbytes <= 0:
            raise ValueError("too many levels")
        arr = (_lib.GemvProblem * len(probs))(*probs)
        size_arr = (ctypes.c_int32 * n)(*sizes)
        self._host = ctypes.create_string_buffer(nbytes)
        st = lib.aqlm_gemv_step_plan(arr, size_arr, n, fmt[0], fmt[1], fmt[2], ctypes.addressof(self._host), nbytes)
        _check(st, "aqlm_gemv_step_plan")
        dev = keep[0][0].device if device is None else device
        self._dev = torch.frombuffer(bytearray(self._host.raw), dtype=torch.uint8).to(dev)
        self.sync = torch.zeros(_lib.STEP_SYNC_BYTES // 4, dtype=torch.int32, device=dev)
        self._keep = keep
        self.levels = n

    def run(self, *, spin_limit: int = 0, stream=None):
        """Launch the step (asynchronous); ``spin_limit`` bounds each level
        barrier's polls (0: the library default)."""
        import ctypes
        st = _lib.load().aqlm_gemv_step(ctypes.addressof(self._host), self._dev.data_ptr(), self.sync.data_ptr(),
                                        int(spin_limit), _stream_handle(stream))
        _check(st, "aqlm_gemv_step")

    def status(self, stream=None):
        """Synchronize and raise AqlmError(AQLM_ERR_TIMEOUT) if a level barrier
        of an earlier run gave up (the flag is cleared)."""
        _check(_lib.load().aqlm_gemv_step_status(self.sync.data_ptr(), _stream_handle(stream)),
               "aqlm_gemv_step_status")


class SortedCodes:
    """Chunk-sorted copy of a layer's codes for the matrix-vector product
    (``aqlm_sort_codes`` / ``aqlm_gemv_sorted``).

    For one or two codebooks of 2^15 or 2^16 codewords: the codes of every
    16-row block are regrouped by 8192-codeword chunk on the host, once, and
    the entries, their index and a zeroed workspace are kept on the layer's
    device.  :meth:`gemv` then computes what :func:`gemv` computes for the
    original codes.  ``codes``: the layer's codes as for :func:`gemv`
    (uint16/int16 [d_out, d_in/8, M], or bit-packed int32 with ``d_in``).
    Calls on one stream may share the object; calls on several streams at
    once need one object each (the workspace is shared)."""

    def __init__(self, codes, codebooks, scales, *, d_in=None):
        d_out, d_in, M, B, g = _args(codes, codebooks, scales, d_in)
        lib = _lib.load()
        host = codes.detach().to("cpu").contiguous()
        ew, iw = ctypes.c_int64(0), ctypes.c_int64(0)
        _check(lib.aqlm_sort_codes_size(host.data_ptr(), d_out, d_in, M, B, g, ctypes.byref(ew),
                                        ctypes.byref(iw)), "aqlm_sort_codes_size")
        entries = torch.empty(ew.value, dtype=torch.int32)
        index = torch.empty(iw.value, dtype=torch.int32)
        _check(lib.aqlm_sort_codes(host.data_ptr(), d_out, d_in, M, B, g, entries.data_ptr(), ew.value,
                                   index.data_ptr(), iw.value), "aqlm_sort_codes")
        dev = codes.device
        self.entries = entries.to(dev)
        self.index = index.to(dev)
        self.index_host = index  # (lets a launch carry the workgroups' first steps)
        self.codebooks, self.scales = codebooks, scales
        self.d_out, self.d_in, self.M, self.B, self.g = d_out, d_in, M, B & ~_lib.PACKED, g
        need = int(lib.aqlm_gemv_sorted_workspace_bytes(d_out, M, self.B))
        # (zero counters before the first launch; launches keep them consistent)
        self.workspace = torch.zeros((need,), dtype=torch.uint8, device=dev)

    def gemv(self, x, *, out=None, stream=None) -> torch.Tensor:
        """y = W x for x fp16 [d_in] on the GPU (as :func:`gemv`)."""
        if x.dtype != torch.float16 or x.numel() != self.d_in or not x.is_cuda or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 GPU tensor with d_in elements")
        out = _out(out, (self.d_out,), self.entries)
        st = _lib.load().aqlm_gemv_sorted(
            self.entries.data_ptr(), self.entries.numel(), self.index.data_ptr(), self.index_host.data_ptr(),
            self.codebooks.data_ptr(),
            self.scales.data_ptr(), self.d_out, self.d_in, self.M, self.B, self.g, x.data_ptr(), out.data_ptr(),
            self.workspace.data_ptr(), self.workspace.numel(), _stream_handle(stream))
        _check(st, "aqlm_gemv_sorted")
        return out


_sorted_ws = {}


def _sorted_workspace(device, need: int) -> torch.Tensor:
    """A zeroed workspace of at least ``need`` bytes for grouped sorted
    launches on ``device`` (kept and grown between calls)."""
    ws = _sorted_ws.get(device)
    if ws is None or ws.numel() < need:
        ws = torch.zeros((need,), dtype=torch.uint8, device=device)
        _sorted_ws[device] = ws
    return ws


def gemv_sorted_grouped(problems, *, workspace=None, stream=None):
    """Several sorted products of one format in one launch
    (``aqlm_gemv_sorted_grouped``): ``problems`` is a list of
    (:class:`SortedCodes`, x fp16 [d_in], y fp16 [d_out]) on one GPU.  Without
    ``workspace`` a zeroed one kept per device is used (calls on several
    streams at once need their own)."""
    if not 1 <= len(problems) <= _lib.MAX_GROUPED:
        raise ValueError(f"1..{_lib.MAX_GROUPED} problems")
    first = problems[0][0]
    arr = (_lib.SortedProblem * len(problems))()
    rows = 0
    for k, (sc, x, y) in enumerate(problems):
        if (sc.M, sc.B, sc.g) != (first.M, first.B, first.g):
            raise ValueError("grouped problems must share (M, B, g)")
        if x.dtype != torch.float16 or x.numel() != sc.d_in or not x.is_cuda or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 GPU tensor with d_in elements")
        _out(y, (sc.d_out,), sc.entries)
        arr[k] = _lib.SortedProblem(sc.entries.data_ptr(), sc.entries.numel(), sc.index.data_ptr(),
                                    sc.index_host.data_ptr(), sc.codebooks.data_ptr(), sc.scales.data_ptr(), x.data_ptr(), y.data_ptr(),
                                    sc.d_out, sc.d_in)
        rows += sc.d_out
    lib = _lib.load()
    need = int(lib.aqlm_gemv_sorted_workspace_bytes(rows, first.M, first.B))
    if workspace is None:
        workspace = _sorted_workspace(first.entries.device, need)
    st = lib.aqlm_gemv_sorted_grouped(arr, len(problems), first.M, first.B, first.g, workspace.data_ptr(),
                                      workspace.numel() * workspace.element_size(), _stream_handle(stream))
    _check(st, "aqlm_gemv_sorted_grouped")
