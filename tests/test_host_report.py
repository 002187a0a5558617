"""Host-side reporting: the paper's speedup percentages reproduce from its timings."""
import os

import numpy as np
import pytest

from paper_2608_27888_amd.report import divergence_metric, paper_speedup_percent

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_timings.txt")


def _load():
    rows, foot = [], []
    for line in open(GOLDEN):
        if not line.strip() or line.startswith("#"):
            continue
        f = line.split()
        if f[0] == "footer":
            foot.append((int(f[1]), float(f[2]), float(f[3]), float(f[4])))
        else:
            rows.append((int(f[1]), int(f[2]), float(f[3]), float(f[4]), float(f[5]), float(f[6])))
    return rows, foot


def test_footers_reproduce_from_table_rows():
    rows, foot = _load()
    assert len(rows) == 20 and len(foot) == 4
    for dec, clk, wmma, fma in foot:
        sel = [r for r in rows if r[0] == dec and r[2] == clk]
        assert len(sel) == 5
        s = [r[3] for r in sel]
        assert paper_speedup_percent(s, [r[4] for r in sel]) == pytest.approx(wmma, abs=0.006)
        assert paper_speedup_percent(s, [r[5] for r in sel]) == pytest.approx(fma, abs=0.006)


def test_abstract_headline_is_mean_ratio_minus_one():
    rows, _ = _load()
    sel = [r for r in rows if r[0] == 10 and r[2] == 1.6]
    ratio = np.mean([r[4] / r[3] for r in sel])
    assert ratio == pytest.approx(9.4849, abs=1e-3)  # "up to 8.48x" = 848.49 % speedup


def test_divergence_metric():
    assert divergence_metric([10, 10, 0, 1]) == 0.0
    assert divergence_metric([4, 10, 3, 4]) == pytest.approx(1.5)
    assert divergence_metric([0, 0, 0, 0]) == 0.0
