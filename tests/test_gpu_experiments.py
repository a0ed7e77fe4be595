"""The paper's synthetic claim on the erase approximation (Sec. 2, Approximate
erasure rate), run on the library's entry points (kda_weights,
kda_weights_exact, kda_alloc_bits): with diverse keys the diagonal
approximation's allocation stays within 3 % of the exact-Gramian allocation's
distortion; with a persistent key it is clearly worse (errors orthogonal to a
repeated key are never erased)."""
import numpy as np
import pytest

from paper_2609_30950_amd import experiments
from tests._gpu import say

pytestmark = pytest.mark.gpu


def test_erase_approximation_diverse_vs_persistent_keys():
    div = experiments.erase_approximation(heads=16, window=256, mean_bits=2.0, keys="diverse",
                                          beta_mode="half")
    per = experiments.erase_approximation(heads=16, window=256, mean_bits=2.0,
                                          keys="persistent", beta_mode="half")
    say(f"excess distortion: diverse max {div.max():.4f} mean {div.mean():.4f}; "
        f"persistent max {per.max():.4f} mean {per.mean():.4f}")
    assert np.all(div >= -1e-12) and np.all(per >= -1e-12)   # the exact allocation is optimal
    assert div.max() <= 0.03
    assert per.mean() > 5 * div.mean() and per.max() > 0.05
