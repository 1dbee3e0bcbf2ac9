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


TOL = {"f32": 1e-5, "bf16": 5e-3}
U24 = 2.0 ** -24           # unit roundoff of fp32 (24-bit significand)
U_OUT = {"f32": 0.0, "bf16": 2.0 ** -8}   # unit roundoff of the stored output (bf16: 8-bit significand)


def check_output(got: np.ndarray, ref: np.ndarray, absref: np.ndarray, kmax: int, in_dt: str, out_dt: str,
                 name: str = "", plane_axes: int = 2) -> float:
    """The parity gates of one forward output against the fp64 oracle.

    * every value is finite;
    * global rel-L2 <= TOL[in_dt] (the stated tolerance);
    * per plane rel-L2 <= TOL[in_dt]: a plane is one (image, output channel) of a
      conv (the last two axes) or one output feature of a linear layer (the last
      axis); an all-zero reference plane must come out exactly zero;
    * element-wise: |got - ref| <= u_out * |ref| + (1 + u_out) * g * absref, where
      absref = sum of |w * x| (+ |bias|) over the kept terms (the oracle run on
      absolute values), g = 2 (kmax + 2) * 2^-24 bounds fp32 accumulation (and the
      products of fp32 inputs) in any summation order with a factor 2 of margin, and
      u_out = 2^-8 is the rounding of a bf16 output (0 for fp32).  Removed weights
      enter the kernel as exact zeros and add nothing to the error.
    A localised mistake (one dropped or mis-decoded kept column, one wrong tile)
    fails the last two even when the global norm hides it.  Returns the global
    rel-L2."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape == absref.shape, (name, got.shape, ref.shape, absref.shape)
    assert np.isfinite(got).all(), f"{name}: {int((~np.isfinite(got)).sum())} non-finite outputs"
    tol = TOL[in_dt]
    err = rel_l2(got, ref)
    assert err <= tol, f"{name}: rel-L2 {err:.3e} > {tol:g}"
    # per plane
    lead = got.shape[:got.ndim - plane_axes] if plane_axes else got.shape
    g2 = got.reshape(int(np.prod(lead)), -1)
    r2 = ref.reshape(g2.shape)
    num = np.linalg.norm(g2 - r2, axis=1)
    den = np.linalg.norm(r2, axis=1)
    zero = den == 0
    assert np.all(num[zero] == 0), f"{name}: {int((num[zero] > 0).sum())} all-zero planes come out nonzero"
    pe = num[~zero] / den[~zero]
    if pe.size:
        worst = int(np.argmax(pe))
        assert pe[worst] <= tol, f"{name}: plane rel-L2 {pe[worst]:.3e} > {tol:g} (plane {np.nonzero(~zero)[0][worst]})"
    # element-wise bound
    u = U_OUT[out_dt]
    g = 2.0 * (kmax + 2) * U24
    bound = u * np.abs(ref) + (1.0 + u) * g * absref
    over = np.abs(got - ref) > bound
    if over.any():
        i = np.unravel_index(int(np.argmax(np.abs(got - ref) - bound)), got.shape)
        raise AssertionError(f"{name}: {int(over.sum())} outputs outside the error bound, worst at {i}: "
                             f"got {got[i]!r} ref {ref[i]!r} bound {bound[i]:.3e}")
    return err


def oracle_mask(w_stored: np.ndarray, dtype: str, scheme) -> np.ndarray:
    wg = as_f64(w_stored, dtype).reshape(scheme.rows, scheme.cols)
    return OP.prune_mask(wg, scheme.bh, scheme.bw, scheme.regularity, scheme.rate, getattr(scheme, "khw", 1))


def oracle_conv(x, w, mask, dtype, layer, bias=None, relu=False, images=None, absolute=False) -> np.ndarray:
    """fp64 direct conv on the masked weights for the chosen images; absolute=True
    runs it on |x|, |w| and |bias| without ReLU (the sum of |terms| of every output)."""
    xf = as_f64(x, dtype)
    if images is not None:
        xf = xf[list(images)]
    wm = as_f64(w, dtype).reshape(layer.cout, -1) * mask.reshape(layer.cout, -1)
    wm = wm.reshape(layer.w_shape)
    if absolute:
        xf, wm = np.abs(xf), np.abs(wm)
        bias = None if bias is None else np.abs(np.asarray(bias, dtype=np.float64))
        relu = False
    return direct.conv2d(xf, wm, bias, (layer.sh, layer.sw), (layer.ph, layer.pw), relu=relu)


def oracle_linear(x, w, mask, dtype, bias=None, relu=False, cols=None, absolute=False) -> np.ndarray:
    xf = as_f64(x, dtype)
    if cols is not None:
        xf = xf[:, list(cols)]
    wm = as_f64(w, dtype).reshape(mask.shape) * mask
    if absolute:
        xf, wm = np.abs(xf), np.abs(wm)
        bias = None if bias is None else np.abs(np.asarray(bias, dtype=np.float64))
        relu = False
    return direct.linear(xf, wm, bias, relu=relu)


def gate_conv(got, x, w, mask, in_dt, out_dt, layer, bias=None, relu=False, images=None, name="") -> float:
    """check_output of a conv output against the oracle (images: the sampled images)."""
    ref = oracle_conv(x, w, mask, in_dt, layer, bias=bias, relu=relu, images=images)
    absref = oracle_conv(x, w, mask, in_dt, layer, bias=bias, images=images, absolute=True)
    kmax = int(mask.reshape(layer.cout, -1).sum(axis=1).max())
    return check_output(got, ref, absref, kmax, in_dt, out_dt, name=name or layer.name, plane_axes=2)


def gate_linear(got, x, w, mask, in_dt, out_dt, bias=None, relu=False, cols=None, name="") -> float:
    """check_output of a feature-major linear output [out][batch]: planes are output features."""
    ref = oracle_linear(x, w, mask, in_dt, bias=bias, relu=relu, cols=cols)
    absref = oracle_linear(x, w, mask, in_dt, bias=bias, cols=cols, absolute=True)
    kmax = int(mask.sum(axis=1).max())
    return check_output(got, ref, absref, kmax, in_dt, out_dt, name=name, plane_axes=1)


def out_to_f64(y_stored: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return y_stored.astype(np.float64)
    return bf16_bits_to_f32(y_stored).astype(np.float64)
