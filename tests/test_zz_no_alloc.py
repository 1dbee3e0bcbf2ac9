"""bsp_prune_noalloc (the allocation-free prune) against bsp_prune through the C
ABI: the same masks, bit for bit, on two calls in a row, the second on a smaller
layer (its fixed per-device scratch keeps the first call's contents).  It must
pass alone in a fresh process and after the other tests."""

import numpy as np
import pytest

from synthetic import draw, seed_for, COL, ROW, UNSTRUCTURED, PUNCHED
from tests.helpers import DT, to_dev, oracle_mask

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2111_11581_amd as B
    B.lib()
    return B


def _both(B, scheme, wdt, w):
    import torch
    n = scheme.rows * scheme.cols
    m_ref = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    m_na = torch.full((n,), 9, dtype=torch.uint8, device="cuda")
    B.bsp_prune(scheme, DT[wdt], w, m_ref)
    B.bsp_prune_noalloc(scheme, DT[wdt], w, m_na)
    torch.cuda.synchronize()
    return m_ref.cpu().numpy(), m_na.cpu().numpy()


def test_unstructured_noalloc_equals_prune_on_two_calls_second_smaller(B):
    # (rows, cols, rate, dtype): a C5-size layer, then a smaller one with ties
    cases = [(256, 2304, 4, "bf16"), (100, 77, 3, "f32")]
    for i, (R, C, rate, dt) in enumerate(cases):
        if i == 0:
            w = draw(seed_for(9, 400, 1), (R, C), ("normal", 0, 0.03), dt)
        else:
            w = np.random.default_rng(5).integers(-2, 3, size=(R, C)).astype(np.float32)
        scheme = B.Scheme(R, C, 1, 1, UNSTRUCTURED, rate)
        m_ref, m_na = _both(B, scheme, dt, to_dev(w, dt))
        assert np.array_equal(m_na, m_ref), f"call {i + 1}: {int((m_na != m_ref).sum())} entries differ"
        assert np.array_equal(m_na.reshape(R, C), oracle_mask(w, dt, scheme))
        assert int(m_na.sum()) == -(-R * C // rate)


def test_block_kinds_noalloc_equal_prune(B):
    for R, C, bh, bw, reg, rate, khw in [(512, 4608, 16, 32, COL, 4, 1), (2048, 512, 32, 32, ROW, 2, 1),
                                         (64, 576, 16, 8, PUNCHED, 3, 9)]:
        w = draw(seed_for(9, 410 + R, 1), (R, C), ("normal", 0, 0.05), "bf16")
        scheme = B.Scheme(R, C, bh, bw, reg, rate, khw)
        m_ref, m_na = _both(B, scheme, "bf16", to_dev(w, "bf16"))
        assert np.array_equal(m_na, m_ref)
