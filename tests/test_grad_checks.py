"""The gradient checks of the GPU parity tests can fail where they should.

The oracle's own head gradient at the headline workload's logit scale
(teacher logits of standard deviation about 1.1, uniform labels) is altered
the way a broken logit-gradient epilogue would alter it: the softmax part of
every non-label row dropped, or one 256-row block of vocabulary rows off by
50 %. Both alterations move the tensor's relative Frobenius error by only
about 1 %, so the per-tensor bound alone accepts them; the per-row and
softmax-only-row bounds reject them. The unaltered gradient passes.
"""

import numpy as np
import pytest

import oracle
from tests.grad_checks import assert_grad, assert_grad_rows, non_label_rows


@pytest.fixture(scope="module")
def teacher_grad():
    # one sub-model (the teacher) with d = 64 and the logit scale of the 3072-wide
    # headline teacher: std(l) = sigma * sqrt(d) = 0.02 * sqrt(3072) = 1.11
    T, V, d = 256, 32768, 64
    r = np.random.default_rng(7)
    h = [r.standard_normal((T, d))]
    W = [r.normal(scale=0.02 * np.sqrt(3072.0 / d), size=(V, d))]
    y = r.integers(0, V, size=T)
    _, gW = oracle.backward(h, W, y, [1.0], [0.0])
    return gW[0], y


def test_unaltered_gradient_passes(teacher_grad):
    gW, y = teacher_grad
    out = assert_grad_rows(gW.copy(), gW, "exact", softmax_rows=non_label_rows(gW.shape[0], y))
    assert out["tensor"] == 0.0


def test_small_perturbation_within_bounds_passes(teacher_grad):
    # bf16 rounding of every entry: well inside every bound
    gW, y = teacher_grad
    r = np.random.default_rng(1)
    noisy = gW * (1.0 + r.uniform(-2 ** -8, 2 ** -8, size=gW.shape))
    assert_grad_rows(noisy, gW, "rounded", softmax_rows=non_label_rows(gW.shape[0], y))


def test_zeroed_softmax_rows_rejected(teacher_grad):
    gW, y = teacher_grad
    mask = non_label_rows(gW.shape[0], y)
    bad = gW.copy()
    bad[mask] = 0.0
    assert_grad(bad, gW, "zeroed softmax rows")  # the per-tensor bound alone accepts this
    with pytest.raises(AssertionError):
        assert_grad_rows(bad, gW, "zeroed softmax rows", softmax_rows=mask)
    with pytest.raises(AssertionError):
        assert_grad_rows(bad, gW, "zeroed softmax rows")  # per-row bound alone


def test_block_off_by_half_rejected(teacher_grad):
    gW, y = teacher_grad
    mask = non_label_rows(gW.shape[0], y)
    bad = gW.copy()
    blk = np.zeros_like(mask)
    blk[4096:4352] = True
    bad[blk & mask] *= 1.5
    assert_grad(bad, gW, "block x1.5")  # the per-tensor bound alone accepts this
    with pytest.raises(AssertionError):
        assert_grad_rows(bad, gW, "block x1.5")


def test_single_row_wrong_rejected(teacher_grad):
    gW, y = teacher_grad
    bad = gW.copy()
    bad[20000] *= -1.0
    with pytest.raises(AssertionError):
        assert_grad_rows(bad, gW, "one row negated")
