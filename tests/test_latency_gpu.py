"""Latency model built on the GPU with the library's forward call (Sec. 5.2.1), and
the block-size rule applied to it (Sec. 5.2.2).  Timing is not pinned; the test
checks that every setting is measured and that the selection obeys the rule."""
import pytest

from paper_2111_11581_amd.latency import LatencyModel, measure, select_block_size, sweep_settings

pytestmark = pytest.mark.gpu

COL, ROW = 1, 0


def test_small_sweep_measures_every_setting_and_selection_obeys_rule(tmp_path):
    st = sweep_settings(cin=64, cout=64, h=16, w=16, batch=4, blocks=(8, 16, 0), rates=(4,), regularities=(ROW, COL))
    m = measure(st, reps=3, rounds=2)
    assert len(m.ms) == len(st) and all(v > 0 for v in m.ms.values())
    p = tmp_path / "lm.json"
    m.save(str(p))
    m = LatencyModel.load(str(p))
    layer = st[0]
    for reg in (ROW, COL):
        for beta in (0.0, 0.2, 10.0):
            bh, bw = select_block_size(m, layer, reg, 4, beta)
            whole = [s for s in st if s.regularity == reg and s.bh == 0][0]
            if (bh, bw) != (0, 0):
                s = [x for x in st if x.regularity == reg and x.bh == bh][0]
                assert m.normalized(s) <= (1 + beta) * m.normalized(whole)
                # nothing smaller qualifies
                for x in st:
                    if x.regularity == reg and 0 < x.bh < bh:
                        assert m.normalized(x) > (1 + beta) * m.normalized(whole)
        # a huge beta accepts every block: the finest one is chosen
        assert select_block_size(m, layer, reg, 4, 10.0) == (8, 8)
