"""Shared test helpers: moving seeded host bits to and from the device, and the
oracle's predictions for one layer.  Oracle inputs always come from the seeded
generators, never from the HIP path."""

from __future__ import annotations

import numpy as np

from oracle import direct
from oracle import prune as OP
from synthetic import bf16_bits_to_f32

DT = {"f32": 0, "bf16": 1}


def to_dev(a: np.ndarray, dtype: str, device="cuda"):
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).view(
        torch.bfloat16).to(device)


def from_dev(t, dtype: str) -> np.ndarray:
    import torch
    t = t.detach().cpu()
    if dtype == "f32":
        return t.numpy().astype(np.float32)
    return t.view(torch.int16).numpy().view(np.uint16)


def as_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    return OP.as_f64(a, dtype)


def rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.reshape(-1))
    num = np.linalg.norm((got - ref).reshape(-1))
    return float(num / den) if den > 0 else float(num)


def oracle_mask(w_stored: np.ndarray, dtype: str, scheme) -> np.ndarray:
    wg = as_f64(w_stored, dtype).reshape(scheme.rows, scheme.cols)
    return OP.prune_mask(wg, scheme.bh, scheme.bw, scheme.regularity, scheme.rate, getattr(scheme, "khw", 1))


def oracle_conv(x, w, mask, dtype, layer, bias=None, relu=False, images=None) -> np.ndarray:
    """fp64 direct conv on the masked weights for the chosen images."""
    xf = as_f64(x, dtype)
    if images is not None:
        xf = xf[list(images)]
    wm = as_f64(w, dtype).reshape(layer.cout, -1) * mask.reshape(layer.cout, -1)
    wm = wm.reshape(layer.w_shape)
    return direct.conv2d(xf, wm, bias, (layer.sh, layer.sw), (layer.ph, layer.pw), relu=relu)


def oracle_linear(x, w, mask, dtype, bias=None, relu=False, cols=None) -> np.ndarray:
    xf = as_f64(x, dtype)
    if cols is not None:
        xf = xf[:, list(cols)]
    wm = as_f64(w, dtype).reshape(mask.shape) * mask
    return direct.linear(xf, wm, bias, relu=relu)


def out_to_f64(y_stored: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return y_stored.astype(np.float64)
    return bf16_bits_to_f32(y_stored).astype(np.float64)
