"""Pins of the junction oracle (eq. (1)) against facts it must satisfy, and
planted mistakes in it that those pins must catch.

* brute force: pure-Python loops (``oracle.bruteforce.junction``);
* the backward against central finite differences of the brute-force forward
  and against torch autograd (float64, CPU) of the forward;
* invariants: the rescaled block has the fresh embedding's norm and the
  direction of ``o``; the fresh block is copied exactly; the two channel
  orders are a permutation of each other; the junction is invariant to a
  positive rescaling of ``o``, so its gradient with respect to ``o`` is
  orthogonal to ``o``;
* zero-norm rows.
"""

import math

import numpy as np
import pytest
import torch

from oracle import bruteforce
from oracle import junction as J


def _draw(T, dp, df, seed, o_scale=30.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, dp)) * o_scale, rng.standard_normal((T, df)),
            rng.standard_normal((T, dp + df)))


@pytest.mark.parametrize("prev_first", [True, False])
def test_forward_matches_brute_force(prev_first):
    o, e, _ = _draw(5, 3, 4, 1)
    ref = np.array(bruteforce.junction(o.tolist(), e.tolist(), prev_first))
    np.testing.assert_allclose(J.forward(o, e, prev_first), ref, rtol=1e-13, atol=1e-13)


def _loss_bruteforce(o, e, g_x, prev_first):
    x = bruteforce.junction(o.tolist(), e.tolist(), prev_first)
    return math.fsum(a * b for row_x, row_g in zip(x, g_x.tolist()) for a, b in zip(row_x, row_g))


@pytest.mark.parametrize("prev_first", [True, False])
def test_backward_matches_central_differences(prev_first):
    o, e, g_x = _draw(3, 4, 3, 2, o_scale=3.0)
    g_o, g_e = J.backward(o, e, g_x, prev_first)
    eps = 1e-6
    for arr, grad in ((o, g_o), (e, g_e)):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            lp = _loss_bruteforce(o, e, g_x, prev_first)
            arr[idx] = old - eps
            lm = _loss_bruteforce(o, e, g_x, prev_first)
            arr[idx] = old
            fd[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(grad, fd, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("prev_first", [True, False])
def test_backward_matches_torch_autograd(prev_first):
    o, e, g_x = _draw(7, 16, 24, 3)
    ot = torch.tensor(o, requires_grad=True)
    et = torch.tensor(e, requires_grad=True)
    scaled = ot * (et.norm(dim=1) / ot.norm(dim=1))[:, None]
    x = torch.cat([scaled, et] if prev_first else [et, scaled], dim=1)
    (x * torch.tensor(g_x)).sum().backward()
    g_o, g_e = J.backward(o, e, g_x, prev_first)
    np.testing.assert_allclose(g_o, ot.grad.numpy(), rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(g_e, et.grad.numpy(), rtol=1e-11, atol=1e-13)


def test_invariants():
    o, e, g_x = _draw(9, 12, 20, 4)
    x = J.forward(o, e, prev_first=True)
    o_t, e_part = x[:, :12], x[:, 12:]
    np.testing.assert_array_equal(e_part, e)  # fresh block copied exactly
    np.testing.assert_allclose(np.linalg.norm(o_t, axis=1), np.linalg.norm(e, axis=1), rtol=1e-13)
    cos = (o_t * o).sum(1) / (np.linalg.norm(o_t, axis=1) * np.linalg.norm(o, axis=1))
    np.testing.assert_allclose(cos, 1.0, rtol=1e-13)
    x2 = J.forward(o, e, prev_first=False)
    np.testing.assert_array_equal(x2, np.concatenate([x[:, 12:], x[:, :12]], axis=1))
    np.testing.assert_allclose(J.forward(o * 7.5, e), x, rtol=1e-13)  # scale invariance in o
    g_o, g_e = J.backward(o, e, g_x)
    np.testing.assert_allclose((g_o * o).sum(1), 0.0, atol=1e-12 * np.abs(g_o).sum())
    # the part of g_e beyond the direct gradient is parallel to e
    extra = g_e - g_x[:, 12:]
    cross = extra[:, :, None] * e[:, None, :] - extra[:, None, :] * e[:, :, None]
    assert np.abs(cross).max() <= 1e-12 * (np.abs(extra).max() * np.abs(e).max() + 1)


def test_zero_norm_rows():
    o, e, g_x = _draw(4, 8, 8, 5)
    o[1] = 0.0
    e[2] = 0.0
    x = J.forward(o, e)
    assert np.all(x[1, :8] == 0) and np.all(x[2, :8] == 0)
    g_o, g_e = J.backward(o, e, g_x)
    assert np.all(g_o[1] == 0) and np.all(g_o[2] == 0)
    np.testing.assert_array_equal(g_e[1], g_x[1, 8:])
    np.testing.assert_array_equal(g_e[2], g_x[2, 8:])
    assert np.all(np.isfinite(g_o)) and np.all(np.isfinite(g_e))


# ---------------------------------------------------------------------------
# planted mistakes (patched into the oracle on the CPU only)
# ---------------------------------------------------------------------------

_orig_fwd = J.forward
_orig_bwd = J.backward


def _mut_ratio_inverted(o, e, prev_first=True):
    x = _orig_fwd(o, e, prev_first)
    dp = np.asarray(o).shape[1]
    blk = slice(0, dp) if prev_first else slice(x.shape[1] - dp, None)
    no = np.linalg.norm(o, axis=1)
    ne = np.linalg.norm(e, axis=1)
    x[:, blk] = np.asarray(o) * (no / ne)[:, None]
    return x


def _mut_no_projection(o, e, g_x, prev_first=True):
    g_o, g_e = _orig_bwd(o, e, g_x, prev_first)
    g = g_x[:, :o.shape[1]] if prev_first else g_x[:, g_x.shape[1] - o.shape[1]:]
    s = np.linalg.norm(e, axis=1) / np.linalg.norm(o, axis=1)
    return s[:, None] * g, g_e


def _mut_g_e_direct_only(o, e, g_x, prev_first=True):
    g_o, _ = _orig_bwd(o, e, g_x, prev_first)
    return g_o, (g_x[:, o.shape[1]:] if prev_first else g_x[:, :e.shape[1]]).copy()


def _mut_split_swapped(o, e, g_x, prev_first=True):
    return _orig_bwd(o, e, g_x, not prev_first)


@pytest.mark.parametrize("name,fwd,bwd", [
    ("ratio_inverted", _mut_ratio_inverted, None),
    ("no_projection", None, _mut_no_projection),
    ("g_e_direct_only", None, _mut_g_e_direct_only),
    ("split_swapped", None, _mut_split_swapped),
])
def test_planted_mistake_is_caught(monkeypatch, name, fwd, bwd):
    if fwd is not None:
        monkeypatch.setattr(J, "forward", fwd)
    if bwd is not None:
        monkeypatch.setattr(J, "backward", bwd)
    checks = [lambda: test_forward_matches_brute_force(True),
              lambda: test_backward_matches_central_differences(True),
              lambda: test_backward_matches_torch_autograd(True),
              test_invariants]
    caught = 0
    for c in checks:
        try:
            c()
        except AssertionError:
            caught += 1
    assert caught > 0, f"mutant {name} passed every pin"
