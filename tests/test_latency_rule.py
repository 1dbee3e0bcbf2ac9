"""Rule-based block-size selection over a latency model (Sec. 5.2.2), host logic.

The selection is pinned against hand-made tables whose answer follows from the
rule as stated: normalise each block size's latency by the layer's MACs, accept
it when within (1 + beta) of structured pruning (whole-matrix blocks) at the same
rate, pick the smallest accepted block.
"""
import json

import pytest

from paper_2111_11581_amd.latency import LatencyModel, Setting, select_block_size, sweep_settings

ROW, COL = 0, 1


def _layer(**kw):
    base = dict(cin=256, cout=256, h=56, w=56, kh=3, kw=3, stride=1, pad=1, batch=64, regularity=COL,
                bh=0, bw=0, rate=4)
    base.update(kw)
    return Setting(**base)


def _model(lat_by_block, reg=COL, rate=4, **kw):
    """lat_by_block: {block side (0 = whole): ms}"""
    return LatencyModel([(_layer(regularity=reg, rate=rate, bh=b, bw=b, **kw), ms) for b, ms in lat_by_block.items()])


def test_smallest_block_within_beta_of_structured():
    # structured 1.0 ms; 4x4 is 1.5x slower, 8x8 1.15x, 16x16 1.05x: beta 0.2 accepts 8 and 16 -> 8
    m = _model({0: 1.0, 4: 1.5, 8: 1.15, 16: 1.05, 32: 1.0})
    assert select_block_size(m, _layer(), COL, 4, beta=0.2) == (8, 8)
    # beta 0.1 accepts only 16 and 32 -> 16; beta 0 accepts 32 (equal) -> 32
    assert select_block_size(m, _layer(), COL, 4, beta=0.1) == (16, 16)
    assert select_block_size(m, _layer(), COL, 4, beta=0.0) == (32, 32)
    # beta 1.0 accepts everything -> the finest block
    assert select_block_size(m, _layer(), COL, 4, beta=1.0) == (4, 4)


def test_no_block_within_beta_returns_structured():
    m = _model({0: 1.0, 8: 1.5, 16: 1.3})
    assert select_block_size(m, _layer(), COL, 4, beta=0.2) == (0, 0)


def test_selection_is_monotone_in_beta():
    m = _model({0: 2.0, 4: 3.1, 8: 2.6, 16: 2.3, 32: 2.1, 64: 2.05})
    areas = []
    for beta in (0.0, 0.03, 0.06, 0.16, 0.31, 0.56, 2.0):
        bh, bw = select_block_size(m, _layer(), COL, 4, beta=beta)
        areas.append(256 * 2304 if bh == 0 else bh * bw)
    assert areas == sorted(areas, reverse=True)


def test_other_rates_regularities_and_layers_are_ignored():
    # a fast 4x4 entry at another rate, another regularity and another layer must not be picked
    m = _model({0: 1.0, 16: 1.1})
    m.add(_layer(regularity=COL, rate=8, bh=4, bw=4), 0.1)
    m.add(_layer(regularity=ROW, rate=4, bh=4, bw=4), 0.1)
    m.add(_layer(cin=128, regularity=COL, rate=4, bh=4, bw=4), 0.1)
    assert select_block_size(m, _layer(), COL, 4, beta=0.2) == (16, 16)


def test_normalisation_by_macs_is_per_layer():
    # the same latencies on a layer with twice the MACs normalise to half: the choice
    # inside one layer does not change (normalisation divides every candidate alike)
    lat = {0: 1.0, 8: 1.15, 16: 1.05}
    a = _model(lat)
    b = _model(lat, h=112, w=112)
    assert select_block_size(a, _layer(), COL, 4, 0.2) == select_block_size(b, _layer(h=112, w=112), COL, 4, 0.2)
    s = _layer(bh=8, bw=8)
    assert a.normalized(s) == pytest.approx(1.15 / s.macs())


def test_missing_structured_entry_raises():
    m = _model({8: 1.0, 16: 1.1})
    with pytest.raises(KeyError):
        select_block_size(m, _layer(), COL, 4, 0.2)


def test_save_load_roundtrip(tmp_path):
    m = _model({0: 1.0, 8: 1.15})
    m.meta["device"] = "test"
    p = tmp_path / "m.json"
    m.save(str(p))
    d = json.loads(p.read_text())
    assert d["meta"]["device"] == "test" and len(d["entries"]) == 2
    m2 = LatencyModel.load(str(p))
    assert m2.ms == m.ms and select_block_size(m2, _layer(), COL, 4, 0.2) == (8, 8)


def test_sweep_settings_cover_the_block_size_sweep():
    st = sweep_settings()
    # 6 block sizes (4..64 and whole) x 3 regularities (row, column, block-punched) x 4 rates,
    # one 3x3 256->256 56x56 b64 layer
    assert len(st) == 72 and len({s.key() for s in st}) == 72
    assert {s.bh for s in st} == {4, 8, 16, 32, 64, 0} and {s.rate for s in st} == {2, 4, 8, 16}
    assert all(s.ho == 56 and s.wo == 56 for s in st)
    assert st[0].macs() == 64 * 256 * 56 * 56 * 256 * 9
    # with the reference points: unstructured at each rate and the dense layer, all distinct
    sr = sweep_settings(references=True)
    assert len(sr) == 81 and len({s.key() for s in sr}) == 81
    assert sorted(s.rate for s in sr if s.regularity == 6) == [2, 4, 8, 16]
    assert sorted(s.rate for s in sr if s.regularity == 2) == [2, 4, 8, 16]
    assert [s.rate for s in sr if s.regularity == 3] == [1]


def test_invalid_latency_rejected():
    with pytest.raises(ValueError):
        LatencyModel([(_layer(), 0.0)])


def test_block_punched_blocks_are_filters_by_channels():
    # a punched block of bh filters x bw channels holds bh * bw kernels of kh*kw weights
    s = Setting(256, 128, 56, 56, 3, 3, 1, 1, 64, 4, 16, 8, 4)
    assert s.area() == 16 * 8 * 9 and "punched 16x8 r4" in s.key()
    assert Setting(256, 128, 56, 56, 3, 3, 1, 1, 64, 4, 0, 0, 4).area() == 128 * 256 * 9


def test_network_settings_cover_every_distinct_layer():
    from paper_2111_11581_amd.latency import network_settings
    layers = [(64, 64, 56, 56, 1, 1, 64), (64, 64, 56, 56, 3, 1, 64), (64, 64, 56, 56, 1, 1, 64),
              (256, 512, 56, 56, 1, 2, 64)]
    st = network_settings(layers, blocks=(8, 0), rates=(4,))
    # 1x1: row and column; 3x3 also block-punched; repeated shapes once
    assert len(st) == 2 * 2 + 3 * 2 + 2 * 2
    assert {s.layer_key() for s in st} == {"1x1/1 64->64 56x56 b64", "3x3/1 64->64 56x56 b64",
                                          "1x1/2 256->512 56x56 b64"}
    assert all(s.pad == s.kh // 2 for s in st)
    assert {s.regularity for s in st if s.kh == 3} == {0, 1, 4}


def test_kept_fraction_from_the_scheme_and_roofline_bound():
    # kept groups per block are ceil(extent / rate) (Sec. 4.1.1): a 4-column block keeps
    # 1 at 4x, 8x and 16x alike; a ragged last block keeps ceil(its width / rate)
    from paper_2111_11581_amd.latency import kept_fraction, roofline
    col44 = [Setting(256, 256, 56, 56, 3, 3, 1, 1, 64, 1, 4, 4, r) for r in (2, 4, 8, 16)]
    assert [kept_fraction(s) for s in col44] == [0.5, 0.25, 0.25, 0.25]
    # 10 columns in blocks of 4: 4 + 4 + 2 -> at 4x keep 1 + 1 + 1 of 10
    assert kept_fraction(Setting(10, 8, 1, 1, 1, 1, 1, 0, 1, 1, 8, 4, 4)) == 3 / 10
    # rows of 20 in blocks of 8 (8 + 8 + 4) at 3x keep 3 + 3 + 2 of 20
    assert kept_fraction(Setting(10, 20, 1, 1, 1, 1, 1, 0, 1, 0, 8, 8, 3)) == 8 / 20
    # block-punched at 4x keeps ceil(9 / 4) = 3 of 9 kernel locations
    assert kept_fraction(Setting(64, 64, 8, 8, 3, 3, 1, 1, 1, 4, 16, 8, 4)) == 3 / 9
    dense = Setting(256, 256, 56, 56, 3, 3, 1, 1, 64, 3, 0, 0, 1)
    assert kept_fraction(dense) == 1.0
    # dense 3x3 256->256 56x56 b64: 2 * 64 * 256 * 56 * 56 * 2304 flops at 2.5166 PFLOP/s
    # is 94.1 us (MFMA-bound: the bytes take 13.2 us at 8 TB/s)
    t_roof = 2.0 * 64 * 256 * 56 * 56 * 2304 / 2.5166e15
    f, bound = roofline(dense, t_roof * 1e3 * 2)
    assert bound == "mfma" and abs(f - 0.5) < 1e-12
