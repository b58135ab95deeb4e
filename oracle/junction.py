"""Float64 CPU oracle of the inter-model junction, forward and backward.

TEST INFRASTRUCTURE ONLY. The product path never imports this module; only
``tests/``, the smoke check and the CPU-baseline leg of ``bench.py`` do.

What is computed (paper section 2, paragraph "Inter-model Junction", eq. (1)):
the output ``o`` of sub-model ``m`` (width ``D_m``) is rescaled so that its
Euclidean norm equals that of the fresh input embedding ``e`` of sub-model
``m+1`` (width ``D_{m+1} - D_m``), and the two are concatenated into the
``D_{m+1}``-wide input of sub-model ``m+1``. The junction has no parameters.

    o_tilde = o * ||e|| / ||o||                     (per token)
    x       = concat(o_tilde, e)   or   concat(e, o_tilde)

Readings taken where the paper is ambiguous or silent:

* Channel order. Eq. (1) writes ``concat(e, o_tilde)``, while the sentence
  after it places sub-model ``m``'s information in the first ``D_m`` channels
  and the fresh embedding in the remaining ones, which is also what nested
  weights (sub-model ``m``'s parameters are the leading block of sub-model
  ``m+1``'s) need. ``prev_first=True`` (the default) follows the sentence,
  ``prev_first=False`` the equation's literal order.
* Zero norms. With ``||o|| = 0`` or ``||e|| = 0`` the rescaled part is 0 and
  every gradient term through the ratio is 0 (the ratio's derivative is taken
  as 0 where a norm vanishes).

Backward, for an upstream gradient ``g_x`` split into ``g`` (the ``o_tilde``
channels) and ``g_e_direct`` (the ``e`` channels), with ``s = ||e|| / ||o||``:

    dL/do = s * (g - (g . o) o / ||o||^2)
    dL/de = g_e_direct + (g . o) / ||o|| * e / ||e||

These are the chain rule of the two lines above; the finite-difference and
autograd pins in ``tests/test_junction_oracle.py`` check them.
"""

from __future__ import annotations

import numpy as np


def _rows(x):
    return np.asarray(x, dtype=np.float64)


def _split(x, d_prev, prev_first):
    """The (o_tilde, e) channel blocks of a junction-output-shaped array."""
    if prev_first:
        return x[:, :d_prev], x[:, d_prev:]
    d_fresh = x.shape[1] - d_prev
    return x[:, d_fresh:], x[:, :d_fresh]


def forward(o, e, prev_first=True):
    """Eq. (1), first line and the concatenation: returns ``x [T, D_prev + D_fresh]``."""
    o = _rows(o)
    e = _rows(e)
    assert o.ndim == 2 and e.ndim == 2 and o.shape[0] == e.shape[0]
    no = np.sqrt((o * o).sum(axis=1))
    ne = np.sqrt((e * e).sum(axis=1))
    ok = (no > 0) & (ne > 0)
    scale = np.where(ok, ne / np.where(no > 0, no, 1.0), 0.0)
    o_t = o * scale[:, None]
    return np.concatenate([o_t, e] if prev_first else [e, o_t], axis=1)


def backward(o, e, g_x, prev_first=True):
    """Gradient of ``L = sum(g_x * x)`` with respect to ``o`` and ``e``: ``(g_o, g_e)``."""
    o = _rows(o)
    e = _rows(e)
    g_x = _rows(g_x)
    g, g_e_direct = _split(g_x, o.shape[1], prev_first)
    no = np.sqrt((o * o).sum(axis=1))
    ne = np.sqrt((e * e).sum(axis=1))
    ok = (no > 0) & (ne > 0)
    safe_no = np.where(ok, no, 1.0)
    safe_ne = np.where(ok, ne, 1.0)
    s = np.where(ok, ne / safe_no, 0.0)
    go = (g * o).sum(axis=1)
    g_o = s[:, None] * (g - (go / safe_no ** 2)[:, None] * o)
    g_o[~ok] = 0.0
    g_e = g_e_direct + np.where(ok, go / safe_no, 0.0)[:, None] * e / safe_ne[:, None]
    return g_o, g_e

