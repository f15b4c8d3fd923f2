"""The parity helper's tie rule, on hand-made results (CPU only).

A row whose first code mismatch sits at an oracle pre-rounding value within 1e-5 code units of a
half-integer is a rounding tie; the columns from there on are left out of the code metrics.  Any
other first mismatch counts in full, including one 6e-4 code units from the half (the size of a
Block-GD step whose sign flipped at lr 3e-6)."""
import types

import numpy as np

from tests import parity as P


class _Gpu:
    def __init__(self, codes, scales, zeros, W):
        class T:
            def __init__(self, a):
                self.a = a

            def cpu(self):
                return self

            def numpy(self):
                return self.a
        self.codes, self.scales, self.zeros, self.W_hat = T(codes), T(scales), T(zeros), T(W)


def _case():
    rng = np.random.default_rng(0)
    m, n = 4, 256
    pre = rng.uniform(0.6, 14.4, size=(m, n))
    pre[1, 70] = 8.4999989          # a tie
    pre[2, 40] = 6.25               # not a tie
    pre[3, 90] = 3.5006             # a sign-flipped Block-GD step, not a tie
    codes = np.clip(np.rint(pre), 0, 15).astype(np.uint8)
    ora = types.SimpleNamespace(codes=codes.copy(), prerounding=pre, scales=np.ones((m, 2), np.float32),
                                zeros=np.full((m, 2), 8, np.uint8), W_hat=np.zeros((m, n)))
    g = codes.copy()
    g[1, 70] += 1                   # other side of the tie, then a cascade over the rest of the row
    g[1, 71::3] ^= 1
    g[2, 40] += 1                   # a real disagreement
    g[3, 90] -= 1                   # the other side of the flipped step
    scales = ora.scales.copy()
    scales[1, 1] = 2.0              # the group after the tie was searched on different weights
    ora.search_margin = np.full((m, 2), np.inf)
    ora.search_margin[0, 1] = 3e-7  # a search near-tie that the GPU decides the other way
    scales[0, 1] = 1.5
    return _Gpu(g, scales, ora.zeros.copy(), ora.W_hat.copy()), ora


def test_tie_cascade_is_found_and_left_out():
    g, ora = _case()
    ties = P.tie_cascades(g.codes.numpy(), ora)
    assert ties == {1: 70}
    met = P.compare(g, ora, tie_cascade=True)
    assert met["tie_cascade_rows"] == 1
    assert met["code_mismatches"] == 2                     # rows 2 and 3 count
    assert met["tie_cascade_codes"] == 1 + len(range(71, 256, 3))
    assert met["group_param_agreement"] == 6 / 7           # group 1 of row 1 is past the tie
    assert met["search_near_ties"] == 1 and met["group_mismatch_at_near_ties"] == 1


def test_tie_window():
    g, ora = _case()
    ora.prerounding[1, 70] = 8.49998            # 2e-5 from the half: outside the window
    assert P.tie_cascades(g.codes.numpy(), ora) == {}


def test_tile_rows_cover_every_tile():
    rows = P.tile_rows(1000, per_tile=1, extra=10, seed=3)
    assert len(rows) == 4 + 10 and len(set(rows)) == len(rows)
    assert set(rows // 256) == {0, 1, 2, 3}


def test_without_the_rule_every_mismatch_counts():
    g, ora = _case()
    met = P.compare(g, ora)
    assert met["tie_cascade_rows"] == 0
    assert met["code_mismatches"] == 3 + len(range(71, 256, 3))
    assert met["group_param_agreement"] < 1.0
