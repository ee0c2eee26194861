"""Host-side pieces of the error controls, on the CPU: Appendix E's
coefficient-growth heuristic GQ_chi worked by hand on Strassen and the
cubic algorithm, and the tie-aware Spearman correlation on a small case."""
import math
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_26077_amd", "libfmm8.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libfmm8.so not built")


def test_gq_chi_by_hand():
    """Strassen: rescaling to unit |U_r|, |V_r| multiplies W_r by
    (2, sqrt2, sqrt2, sqrt2, sqrt2, 2, 2); chi^A + chi^B per term is
    (2, 1, 1, 1, 1, 2, 2) (M3, M4 have one-entry U_r, M2, M5 one-entry V_r).
    Summing W_rq^2 (chi^A + chi^B) over r gives 20, 4, 4, 20 at C11, C21,
    C12, C22: mean 12, GQ_chi = sqrt(12).  The cubic algorithm's one-entry
    rows give 0, at any shape."""
    from paper_2609_26077_amd import controls, fmm_realization_builtin
    assert controls.gq_chi(fmm_realization_builtin("strassen")) == pytest.approx(math.sqrt(12), rel=1e-15)
    assert controls.gq_chi(fmm_realization_builtin("cubic8")) == 0.0
    assert controls.gq_chi(controls.shaped_realization("cubic_345")) == 0.0


def test_spearman_average_ranks():
    """x = (1, 2, 3, 3) ranks as (1, 2, 3.5, 3.5): against (1, 2, 3, 4) the
    Pearson correlation of the ranks is 4.5 / sqrt(4.5 * 5) = sqrt(0.9)."""
    from paper_2609_26077_amd import controls
    assert controls.spearman([1, 2, 3, 3], [1, 2, 3, 4]) == pytest.approx(math.sqrt(0.9), rel=1e-14)
    assert controls.spearman([3, 1, 2], [30, 10, 20]) == pytest.approx(1.0)
