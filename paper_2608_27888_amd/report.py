"""Host-side reporting helpers (no decode arithmetic).

The paper reports "average speedup" of the shared decoder over non-shared
decoders as a percentage (Sec. 4.4, table footers of the 5- and 10-decoder
timing tables).  Those footers equal the mean over output resolutions of
(T_nonshared / T_shared - 1) x 100, which is the form reproduced here so that
MI355X ratios can be quoted next to the paper's.
"""
from __future__ import annotations

import numpy as np


def paper_speedup_percent(t_shared, t_nonshared) -> float:
    """Mean of (T_nonshared / T_shared - 1) x 100 over paired timings."""
    a = np.asarray(t_shared, dtype=np.float64)
    b = np.asarray(t_nonshared, dtype=np.float64)
    return float(np.mean(b / a - 1.0) * 100.0)


def divergence_metric(totals) -> float:
    """Mean excess of the per-window distinct count over one (Eq. normalized_ones_metric),
    from the totals [windows, sum of distinct counts, divergent windows, max]."""
    n = int(totals[0])
    return 0.0 if n == 0 else float(totals[1]) / n - 1.0
