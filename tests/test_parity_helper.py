"""The parity helper's tie rule, on hand-made results (CPU only).

A row whose first code mismatch sits at an oracle pre-rounding value within 1e-3 code units of a
half-integer is a rounding tie; the columns from there on are left out of the code metrics.  Any
other first mismatch counts in full."""
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
    codes = np.clip(np.rint(pre), 0, 15).astype(np.uint8)
    ora = types.SimpleNamespace(codes=codes.copy(), prerounding=pre, scales=np.ones((m, 2), np.float32),
                                zeros=np.full((m, 2), 8, np.uint8), W_hat=np.zeros((m, n)))
    g = codes.copy()
    g[1, 70] += 1                   # other side of the tie, then a cascade over the rest of the row
    g[1, 71::3] ^= 1
    g[2, 40] += 1                   # a real disagreement
    scales = ora.scales.copy()
    scales[1, 1] = 2.0              # the group after the tie was searched on different weights
    return _Gpu(g, scales, ora.zeros.copy(), ora.W_hat.copy()), ora


def test_tie_cascade_is_found_and_left_out():
    g, ora = _case()
    ties = P.tie_cascades(g.codes.numpy(), ora)
    assert ties == {1: 70}
    met = P.compare(g, ora, tie_cascade=True)
    assert met["tie_cascade_rows"] == 1
    assert met["code_mismatches"] == 1                     # only row 2's disagreement counts
    assert met["tie_cascade_codes"] == 1 + len(range(71, 256, 3))
    assert met["group_param_agreement"] == 1.0             # group 1 of row 1 is past the tie


def test_without_the_rule_every_mismatch_counts():
    g, ora = _case()
    met = P.compare(g, ora)
    assert met["tie_cascade_rows"] == 0
    assert met["code_mismatches"] == 2 + len(range(71, 256, 3))
    assert met["group_param_agreement"] < 1.0
