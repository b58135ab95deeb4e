"""Gradient comparisons shared by the GPU parity tests (pure numpy, no GPU).

A single relative Frobenius bound per tensor is dominated by the largest
entries. In the head gradient ``grad_W_i = G_i^T h_i`` those are the rows of
the tokens' labels, where the logit gradient carries the ``-onehot`` term of
the cross-entropy; the softmax part of ``G_i`` (every other vocabulary row,
the part the fused logit-gradient epilogue actually computes) holds only a
few percent of the norm. So besides the per-tensor bound every row is
checked on its own, and the rows that are no valid token's label are
checked together under a separate relative bound.
"""

from __future__ import annotations

import numpy as np

GRAD_RTOL = 2e-2      # relative Frobenius bound per tensor, per row, and on the softmax-only rows
# Absolute floor of the per-row bound, as a fraction of the median row norm. It
# matters only for rows whose logit gradient nearly cancels (e.g. with two
# vocabulary entries, p - (1 - alpha) onehot - alpha q can be far below its
# terms): there the rounding of the terms (the slab's bf16, the teacher's q)
# is absolute, a few 1e-4 of a typical row, not relative to the small result.
ROW_FLOOR = 5e-3


def rel_fro(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def assert_grad(g, ref, what="", rtol=GRAD_RTOL):
    """Per-tensor bound only: ``||g - ref||_F <= rtol ||ref||_F``."""
    assert np.all(np.isfinite(g)), f"{what}: non-finite gradient"
    if g.ndim == 2 and g.shape[0] > 16384:
        e_r, n_r = row_errors(g, ref)
        nr = np.sqrt((n_r ** 2).sum())
        err = np.sqrt((e_r ** 2).sum()) / (nr if nr > 0 else 1.0)
    else:
        err = rel_fro(g, ref)
    assert err <= rtol, f"{what}: relative Frobenius error {err:.3e} > {rtol}"
    return err


def row_errors(g, ref, block=16384):
    """Per-row error and reference norms (float64, a block of rows at a time)."""
    n = g.shape[0]
    e = np.empty(n)
    r = np.empty(n)
    for b in range(0, n, block):
        gb = np.asarray(g[b:b + block], dtype=np.float64)
        rb = np.asarray(ref[b:b + block], dtype=np.float64)
        e[b:b + block] = np.linalg.norm(gb - rb, axis=1)
        r[b:b + block] = np.linalg.norm(rb, axis=1)
    return e, r


def assert_grad_rows(g, ref, what="", rtol=GRAD_RTOL, softmax_rows=None):
    """Per-tensor, per-row and (optionally) softmax-only-row bounds.

    * the whole tensor: ``||g - ref||_F <= rtol ||ref||_F``;
    * every row r: ``||g_r - ref_r|| <= rtol ||ref_r|| + ROW_FLOOR * median_r ||ref_r||``
      (the floor only matters for rows whose reference is far below the typical row);
    * ``softmax_rows`` (a boolean mask or index array over the rows, e.g. the
      vocabulary rows that are no valid token's label): their joint relative
      Frobenius error is at most rtol.
    Returns a dict of the observed errors.
    """
    assert g.shape == ref.shape, f"{what}: shape {g.shape} != {ref.shape}"
    err = assert_grad(g, ref, what, rtol)
    e_r, n_r = row_errors(g, ref)
    pos = n_r[n_r > 0]
    floor = ROW_FLOOR * (np.median(pos) if pos.size else 0.0)
    bound = rtol * n_r + floor
    bad = np.flatnonzero(e_r > bound)
    if bad.size:
        r = bad[np.argmax(e_r[bad] / np.maximum(bound[bad], 1e-300))]
        raise AssertionError(
            f"{what}: {bad.size} of {len(n_r)} rows exceed the per-row bound; worst row {r}: "
            f"error {e_r[r]:.3e}, reference norm {n_r[r]:.3e}, bound {bound[r]:.3e}")
    worst_row = float(np.max(e_r / np.maximum(n_r, 1e-300), initial=0.0)) if n_r.size else 0.0
    out = {"tensor": err, "worst_row": worst_row}
    if softmax_rows is not None:
        sel = np.zeros(len(n_r), dtype=bool)
        sel[np.asarray(softmax_rows)] = True
        ns = np.sqrt((n_r[sel] ** 2).sum())
        if ns > 0:
            es = np.sqrt((e_r[sel] ** 2).sum()) / ns
            assert es <= rtol, (f"{what}: softmax-only rows relative error {es:.3e} > {rtol}")
            out["softmax_rows"] = es
    return out


def non_label_rows(V, labels, ignore_index=-100):
    """Boolean mask of the vocabulary rows that are no valid token's label."""
    lab = np.asarray(labels)
    lab = lab[(lab != ignore_index) & (lab >= 0) & (lab < V)]
    mask = np.ones(V, dtype=bool)
    mask[lab] = False
    return mask
