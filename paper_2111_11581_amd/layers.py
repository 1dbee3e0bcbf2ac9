"""Convenience wrappers that allocate the library's buffers with torch.

Still argument marshalling only: pruning, packing and the forward run in the
HIP kernels behind the C ABI.
"""

from __future__ import annotations

import torch

from . import (BF16, F32, ConvShape, Scheme, bsp_conv2d, bsp_linear, bsp_pack, bsp_packed_sizes,
               bsp_prune, bsp_unpack)

TORCH_DT = {F32: torch.float32, BF16: torch.bfloat16}


class PackedLayer:
    """Pruned + packed weights of one conv (conv is a ConvShape) or FC (conv None) layer.

    ``w`` is the GEMM-form weight matrix on the device (rows x cols, fp32 or
    bf16).  ``mask`` may be given (it is then validated by bsp_pack);
    otherwise bsp_prune computes it.
    """

    def __init__(self, scheme, wdt: int, w: torch.Tensor, conv=None, mask: torch.Tensor | None = None,
                 stream=None):
        self.scheme = scheme if isinstance(scheme, Scheme) else Scheme(
            scheme.rows, scheme.cols, scheme.bh, scheme.bw, scheme.regularity, scheme.rate,
            getattr(scheme, "khw", 1)).set_counts(getattr(scheme, "counts", None))
        self.wdt = wdt
        self.conv = conv if (conv is None or isinstance(conv, ConvShape)) else ConvShape(*conv)
        dev = w.device
        R, C = self.scheme.rows, self.scheme.cols
        if mask is None:
            mask = torch.empty(R * C, dtype=torch.uint8, device=dev)
            bsp_prune(self.scheme, wdt, w, mask, stream)
        self.mask = mask
        nv, ni, nr, nb = bsp_packed_sizes(self.scheme, self.conv, wdt)
        self.values = torch.empty(max(nv, 1), dtype=TORCH_DT[wdt], device=dev)
        self.indices = torch.empty(max(ni, 1), dtype=torch.int32, device=dev)
        self.rowptr = torch.empty(max(nr, 1), dtype=torch.int32, device=dev)
        self.tiles = torch.empty(nb, dtype=torch.uint8, device=dev)
        self.n_values, self.n_indices, self.n_rowptr = nv, ni, nr
        bsp_pack(self.scheme, wdt, w, mask, self.values, self.indices, self.rowptr, self.tiles,
                 self.conv, stream)

    def unpack(self, stream=None) -> torch.Tensor:
        R, C = self.scheme.rows, self.scheme.cols
        out = torch.empty(R * C, dtype=TORCH_DT[self.wdt], device=self.tiles.device)
        bsp_unpack(self.scheme, self.wdt, self.values, self.indices, self.rowptr, out, stream)
        return out

    def conv2d(self, x, y, n: int, out_dt: int, bias=None, relu=False, stream=None):
        c = self.conv
        shape = ConvShape(n, c.cin, c.h, c.w, c.kh, c.kw, c.stride_h, c.stride_w, c.pad_h, c.pad_w)
        bsp_conv2d(self.scheme, shape, self.wdt, out_dt, x, self.tiles, bias, relu, y, stream)

    def linear(self, x, y, batch: int, out_dt: int, bias=None, relu=False, stream=None):
        bsp_linear(self.scheme, batch, self.wdt, out_dt, x, self.tiles, bias, relu, y, stream)
