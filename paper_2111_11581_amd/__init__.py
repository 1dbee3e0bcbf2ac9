"""Block-structured pruned conv / FC inference on AMD MI355X (gfx950).

Thin ctypes binding of the C ABI in ``include/bsp.h`` (``libbsp.so``, built by
``python -m paper_2111_11581_amd.build``).  The functions below have the same
names as the C entry points and only marshal arguments: torch tensors supply
device pointers, torch's current HIP stream is the default stream.  Every step
of the computation runs in the library's HIP kernels; if the library is not
built, importing the functions raises - there is no fallback.
"""

from __future__ import annotations

import ctypes
import os

__all__ = [
    "F32", "BF16", "ROW", "COL", "UNSTRUCTURED", "DENSE", "PUNCHED", "ROWCOL", "PATTERN", "BspError", "Scheme", "ConvShape",
    "lib", "lib_path", "bsp_packed_sizes", "bsp_prune", "bsp_prune_noalloc", "bsp_pack", "bsp_unpack", "bsp_conv2d",
    "bsp_linear", "bsp_maxpool2x2", "bsp_status_string", "bsp_version", "bsp_to_bcs",
]

F32, BF16 = 0, 1
ROW, COL, UNSTRUCTURED, DENSE, PUNCHED, ROWCOL, PATTERN = 0, 1, 2, 3, 4, 5, 6

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_build", "libbsp.so")
_lib = None


class BspError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {bsp_status_string(status)} ({status})")


class Scheme(ctypes.Structure):
    """bsp_scheme.  ``counts`` (optional) is a host int32 array of kept groups per
    block; set it with ``set_counts`` so that the array outlives the scheme's use."""
    _fields_ = [(n, ctypes.c_int32) for n in ("rows", "cols", "bh", "bw", "regularity", "rate", "khw")] + [
        ("counts", ctypes.POINTER(ctypes.c_int32))]

    def set_counts(self, counts):
        if counts is None:
            self._counts_buf = None
            self.counts = ctypes.POINTER(ctypes.c_int32)()
            return self
        flat = [int(v) for row in counts for v in (row if hasattr(row, "__iter__") else [row])]
        self._counts_buf = (ctypes.c_int32 * len(flat))(*flat)
        self.counts = ctypes.cast(self._counts_buf, ctypes.POINTER(ctypes.c_int32))
        return self


class ConvShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n", "cin", "h", "w", "kh", "kw", "stride_h",
                                               "stride_w", "pad_h", "pad_w")]


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load libbsp.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2111_11581_amd.build`")
    L = ctypes.CDLL(_LIB_PATH)
    P, I32, I64, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    sch, cs = P(Scheme), P(ConvShape)
    L.bsp_packed_sizes.argtypes = [sch, cs, I32, P(I64), P(I64), P(I64), P(I64)]
    L.bsp_prune.argtypes = [sch, I32, VP, VP, VP]
    L.bsp_prune_noalloc.argtypes = [sch, I32, VP, VP, VP]
    L.bsp_pack.argtypes = [sch, I32, VP, VP, VP, VP, VP, VP, cs, VP]
    L.bsp_unpack.argtypes = [sch, I32, VP, VP, VP, VP, VP]
    L.bsp_conv2d.argtypes = [sch, cs, I32, I32, VP, VP, VP, I32, VP, VP]
    L.bsp_linear.argtypes = [sch, I32, I32, I32, VP, VP, VP, I32, VP, VP]
    L.bsp_maxpool2x2.argtypes = [I32, I32, I32, I32, I32, VP, VP, VP]
    L.bsp_status_string.argtypes = [I32]
    L.bsp_status_string.restype = ctypes.c_char_p
    L.bsp_version.argtypes = []
    for f in ("bsp_packed_sizes", "bsp_prune", "bsp_prune_noalloc", "bsp_pack", "bsp_unpack", "bsp_conv2d",
              "bsp_linear", "bsp_maxpool2x2", "bsp_version", "bsp_to_bcs"):
        getattr(L, f).restype = I32
    _lib = L
    return L


def _scheme(s) -> Scheme:
    if isinstance(s, Scheme):
        return s
    out = Scheme(int(s.rows), int(s.cols), int(s.bh), int(s.bw), int(s.regularity), int(s.rate),
                 int(getattr(s, "khw", 1)))
    return out.set_counts(getattr(s, "counts", None))


def _shape(c) -> ConvShape | None:
    if c is None or isinstance(c, ConvShape):
        return c
    return ConvShape(*[int(v) for v in c])


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(getattr(stream, "cuda_stream", stream)))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(fn: str, st: int):
    if st != 0:
        raise BspError(fn, st)


def _need(name: str, t, nbytes: int):
    if t is None:
        raise ValueError(f"{name} is required")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, {nbytes} needed")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def bsp_status_string(status: int) -> str:
    return lib().bsp_status_string(int(status)).decode()


def bsp_version() -> int:
    return int(lib().bsp_version())


def bsp_packed_sizes(scheme, conv, wdt: int):
    """-> (n_values, n_indices, n_rowptr, dev_tile_bytes)."""
    out = [ctypes.c_int64() for _ in range(4)]
    sh = _shape(conv)
    _check("bsp_packed_sizes", lib().bsp_packed_sizes(
        ctypes.byref(_scheme(scheme)), ctypes.byref(sh) if sh is not None else None, int(wdt),
        *[ctypes.byref(o) for o in out]))
    return tuple(int(o.value) for o in out)


def _esize(dt: int) -> int:
    return 4 if dt == F32 else 2


def bsp_prune(scheme, wdt: int, w, mask, stream=None):
    s = _scheme(scheme)
    _need("w", w, s.rows * s.cols * _esize(wdt))
    _need("mask", mask, s.rows * s.cols)
    _check("bsp_prune", lib().bsp_prune(ctypes.byref(s), int(wdt), _p(w), _p(mask), _stream(stream)))


def bsp_prune_noalloc(scheme, wdt: int, w, mask, stream=None):
    s = _scheme(scheme)
    _need("w", w, s.rows * s.cols * _esize(wdt))
    _need("mask", mask, s.rows * s.cols)
    _check("bsp_prune_noalloc", lib().bsp_prune_noalloc(ctypes.byref(s), int(wdt), _p(w), _p(mask),
                                                        _stream(stream)))


def bsp_pack(scheme, wdt: int, w, mask, values, indices, rowptr, dev_tiles, conv=None, stream=None):
    s = _scheme(scheme)
    nv, ni, nr, nb = bsp_packed_sizes(s, conv, wdt)
    _need("w", w, s.rows * s.cols * _esize(wdt))
    _need("mask", mask, s.rows * s.cols)
    _need("values", values, nv * _esize(wdt))
    if ni:
        _need("indices", indices, ni * 4)
    if nr:
        _need("rowptr", rowptr, nr * 4)
    _need("dev_tiles", dev_tiles, nb)
    sh = _shape(conv)
    _check("bsp_pack", lib().bsp_pack(ctypes.byref(s), int(wdt), _p(w), _p(mask), _p(values),
                                      _p(indices), _p(rowptr), _p(dev_tiles),
                                      ctypes.byref(sh) if sh is not None else None, _stream(stream)))


def bsp_unpack(scheme, wdt: int, values, indices, rowptr, w_out, stream=None):
    s = _scheme(scheme)
    _need("w_out", w_out, s.rows * s.cols * _esize(wdt))
    _check("bsp_unpack", lib().bsp_unpack(ctypes.byref(s), int(wdt), _p(values), _p(indices),
                                          _p(rowptr), _p(w_out), _stream(stream)))


def bsp_to_bcs(scheme, indices, rowptr, occurrence, compact_cols, col_stride, row_offset, n_runs, stream=None):
    s = _scheme(scheme)
    _need("row_offset", row_offset, (s.rows + 1) * 4)
    _need("n_runs", n_runs, 4)
    _check("bsp_to_bcs", lib().bsp_to_bcs(ctypes.byref(s), _p(indices), _p(rowptr), _p(occurrence),
                                          _p(compact_cols), _p(col_stride), _p(row_offset), _p(n_runs),
                                          _stream(stream)))


def bsp_conv2d(scheme, shape, in_dt: int, out_dt: int, x, dev_tiles, bias, relu: bool, y, stream=None):
    s, sh = _scheme(scheme), _shape(shape)
    ho = (sh.h + 2 * sh.pad_h - sh.kh) // sh.stride_h + 1
    wo = (sh.w + 2 * sh.pad_w - sh.kw) // sh.stride_w + 1
    _need("x", x, sh.n * sh.cin * sh.h * sh.w * _esize(in_dt))
    _need("y", y, sh.n * s.rows * ho * wo * _esize(out_dt))
    _need("dev_tiles", dev_tiles, bsp_packed_sizes(s, sh, in_dt)[3])
    if bias is not None:
        _need("bias", bias, s.rows * 4)
    _check("bsp_conv2d", lib().bsp_conv2d(ctypes.byref(s), ctypes.byref(sh), int(in_dt), int(out_dt),
                                          _p(x), _p(dev_tiles), _p(bias), int(bool(relu)), _p(y),
                                          _stream(stream)))


def bsp_linear(scheme, batch: int, in_dt: int, out_dt: int, x, dev_tiles, bias, relu: bool, y,
               stream=None):
    s = _scheme(scheme)
    _need("x", x, s.cols * batch * _esize(in_dt))
    _need("y", y, s.rows * batch * _esize(out_dt))
    _need("dev_tiles", dev_tiles, bsp_packed_sizes(s, None, in_dt)[3])
    if bias is not None:
        _need("bias", bias, s.rows * 4)
    _check("bsp_linear", lib().bsp_linear(ctypes.byref(s), int(batch), int(in_dt), int(out_dt), _p(x),
                                          _p(dev_tiles), _p(bias), int(bool(relu)), _p(y),
                                          _stream(stream)))


def bsp_maxpool2x2(dt: int, n: int, c: int, h: int, w: int, x, y, stream=None):
    _need("x", x, n * c * h * w * _esize(dt))
    _need("y", y, n * c * (h // 2) * (w // 2) * _esize(dt))
    _check("bsp_maxpool2x2", lib().bsp_maxpool2x2(int(dt), int(n), int(c), int(h), int(w), _p(x),
                                                  _p(y), _stream(stream)))
