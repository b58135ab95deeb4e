"""The sampled-token check of the GPU decode tests accepts exactly what it
should: tokens the oracle draws within the EPS box (including a swap of equal
probabilities at the nucleus boundary) and no others, up to the allowed count."""

import numpy as np
import pytest

from oracle import decode as OD
from tests.decode_checks import check_samples, oracle_tokens_near


def _boundary_tie_row():
    # p(0) dominates; tokens 1 and 5 tie; top_p halfway between keeping {0} and
    # {0, 1, 5}: the oracle keeps {0, 1} (lower index first), fp32 may keep {0, 5}
    row = np.array([3.0, 0.5, -5.0, -5.0, -5.0, 0.5, -5.0, -5.0])
    p = np.exp(row - row.max())
    p /= p.sum()
    top_p = p[0] + 0.5 * p[1]
    return row, top_p


def test_boundary_swap_accepted_and_other_tokens_rejected():
    row, top_p = _boundary_tie_row()
    u = 0.95  # beyond token 0's share of the kept mass (0.924)
    assert OD.sample(row[None, :], np.array([u]), 1.0, top_p)[0] == 1
    near = oracle_tokens_near(row, u, 1.0, top_p)
    assert near == {1, 5}
    check_samples(row[None, :], np.array([u]), np.array([5]), 1.0, top_p, allowed=1)
    with pytest.raises(AssertionError):  # a token of no kept set
        check_samples(row[None, :], np.array([u]), np.array([3]), 1.0, top_p, allowed=1)
    with pytest.raises(AssertionError):  # a reproducible token beyond the allowed count
        check_samples(row[None, :], np.array([u]), np.array([5]), 1.0, top_p, allowed=0)


def test_uniform_box_reaches_neighbours_only_within_eps():
    rng = np.random.default_rng(4)
    row = rng.standard_normal(3000) * 3.0
    r = OD.filtered_probs(row, 0.7, 0.9)
    cdf = np.cumsum(r)
    v = int(np.nonzero(r > 0)[0][10])  # a kept token (of some 35)
    u_edge = cdf[v] - 0.3e-5          # just below its right edge: the next kept token is within EPS
    nxt = int(np.nonzero(r[v + 1:] > 0)[0][0]) + v + 1
    near = oracle_tokens_near(row, float(u_edge), 0.7, 0.9)
    assert {v, nxt} <= near
    far = oracle_tokens_near(row, float(cdf[v] - 0.5 * r[v]), 0.7, 0.9)  # mid-token: only v
    assert far == {v}
