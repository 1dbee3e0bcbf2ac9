"""Oracle for the glue between VGG stages.  TEST INFRASTRUCTURE ONLY.

2x2 max pooling with stride 2 (floor), NCHW: the standard VGG down-sampling
between stages.  It is not part of the pruning method; the VGG-16 stack
workload needs it between convs.
"""

from __future__ import annotations

import numpy as np


def maxpool2x2(x: np.ndarray) -> np.ndarray:
    N, C, H, W = x.shape
    Ho, Wo = H // 2, W // 2
    out = np.empty((N, C, Ho, Wo), dtype=x.dtype)
    for i in range(Ho):
        for j in range(Wo):
            out[:, :, i, j] = np.maximum(np.maximum(x[:, :, 2 * i, 2 * j], x[:, :, 2 * i, 2 * j + 1]),
                                         np.maximum(x[:, :, 2 * i + 1, 2 * j], x[:, :, 2 * i + 1, 2 * j + 1]))
    return out
