"""Host-side checks of bench.py's threshold handling (no GPU): the offline
threshold search on a synthetic timing table, and the committed thresholds
file the benchmark reads by default."""
import json
import os
from types import SimpleNamespace

import pytest

import bench

ABI = SimpleNamespace(PATH_DENSE_MFMA=0, PATH_SKIP_MFMA=1, PATH_DENSE_BW=2, PATH_SKIP_BW=3)


def _case(m, rho_b_bw, rho_b_mfma, t):
    """t: forced whole-path times (us) per path 0..3."""
    return SimpleNamespace(m=m, inten=dict(intensity={1: 1.0, 8: 7.97, 64: 62.06}[m]),
                           rho_b={2: rho_b_bw, 0: rho_b_mfma}, forced=dict(enumerate(t)))


def _table():
    cases = []
    # m = 1: streaming family wins; its skip path wins from block sparsity 0.5 on
    for rb, t_skip in ((0.0, 16.0), (0.5, 12.0), (0.8, 8.0), (0.95, 4.0)):
        cases.append(_case(1, rb, rb, (30.0, 31.0, 14.0, t_skip)))
    # m = 8: skip wins at 0.8 and 0.95 but not at 0.5 (a gap: no win below 0.8)
    for rb, t_skip in ((0.0, 16.0), (0.5, 14.1), (0.8, 9.0), (0.95, 5.0)):
        cases.append(_case(8, rb, rb, (30.0, 31.0, 14.0, t_skip)))
    # m = 64: the MFMA family is faster; its skip path never wins by 3 %
    for rb in (0.0, 0.5, 0.8, 0.95):
        cases.append(_case(64, rb, rb, (20.0, 19.9, 40.0, 30.0)))
    return cases


def test_calibrate_on_synthetic_timings():
    thr = bench.calibrate(ABI, _table())
    assert thr[1] == (0.5, bench.INTENSITY_THR)
    # 14.1 us is not 3 % below 14.0: the m = 8 class skips only from 0.8
    assert thr[8] == (0.8, bench.INTENSITY_THR)
    # MFMA family: its intensity threshold is the class's own intensity, so
    # the class routes to MFMA; no skip win -> threshold 1.0
    assert thr[64] == (1.0, 62.06)


def test_calibrate_prefers_batched_family_times():
    cases = _table()
    batch = {(m, f): (10.0 if f == ABI.PATH_DENSE_MFMA else 20.0)
             for m in (1, 8, 64) for f in (ABI.PATH_DENSE_BW, ABI.PATH_DENSE_MFMA)}
    thr = bench.calibrate(ABI, cases, batch)
    assert all(thr[m][1] == {1: 1.0, 8: 7.97, 64: 62.06}[m] for m in (1, 8, 64))


def test_load_thresholds_forms(tmp_path):
    obj = {"1": [0.5, 315.0], "8": [0.8, 315.0], "64": [0.9, 62.0]}
    want = {1: (0.5, 315.0), 8: (0.8, 315.0), 64: (0.9, 62.0)}
    assert bench.load_thresholds(json.dumps(obj)) == want
    f = tmp_path / "t.json"
    f.write_text(json.dumps(dict(thresholds_per_m=obj, rule="x")))
    assert bench.load_thresholds(str(f)) == want


def test_committed_thresholds_file():
    if not os.path.exists(bench.THRESHOLDS_FILE):
        pytest.skip("no committed calibration yet")
    thr = bench.load_thresholds(bench.THRESHOLDS_FILE)
    assert sorted(thr) == list(bench.M_LIST)
    for s_thr, c_thr in thr.values():
        assert 0.0 < s_thr <= 1.0 and c_thr > 0.0
