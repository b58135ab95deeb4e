"""Float64 CPU oracle of the Matryoshka multi-head LM loss, forward and backward.

TEST INFRASTRUCTURE ONLY. The product path (the HIP library and its Python
binding) never imports this module; only ``tests/``, the smoke check and the
CPU-baseline leg of ``bench.py`` do.

What is computed (paper: "Matryoshka Language Model Suites", section 2,
"Method"):

* Every nested sub-model ``i`` owns an LM head ``W_i`` of shape ``[V, d_i]``
  and maps its final hidden states ``h_i[t]`` to logits ``l_i[t] = W_i h_i[t]``
  (section 2, paragraphs "Modeling" and "Inter-model Junction").
* Each sub-model is trained with next-token cross-entropy ``CE_i``
  (section 2, "Inter-model Junction", last paragraph).
* Every sub-model other than the largest one (the teacher ``s``) adds a
  distillation term from the teacher's stop-gradient softmax, eq. (2).
* The per-sub-model loss is the convex combination of eq. (3) and the
  training objective is their sum (text after eq. (3)); per-sub-model
  weights follow appendix G ("Closing the Per-Size Gap with Loss
  Weighting").

Readings taken where the paper is silent:

* Temperature ``tau``: the teacher distribution is ``q = softmax(l_s / tau)``
  and the student is ``p_i^tau = softmax(l_i / tau)``; cross-entropy always
  uses ``tau = 1``. With ``tau = 1`` this is eq. (2) exactly.
* The returned distillation value is ``KL(q || p_i^tau)``; eq. (2) itself is
  ``KL + H(q)``, and the teacher entropy ``H(q)`` is returned separately so
  the eq. (2) value is ``KL_i + H``. Both have the same gradient.
* Token reduction is the mean over valid (non-ignored) tokens for every loss;
  with no valid token every loss and gradient is zero.
* ``stop_grad`` in eq. (2) means the teacher receives no gradient from any
  distillation term.
* The loss coefficients ``g_ce[i]``, ``g_kl[i]`` of the objective
  ``J = sum_i g_ce[i] CE_i + g_kl[i] KL_i`` come from :func:`coeffs`; the
  ``tau**2`` factor on the KL term (the usual temperature compensation) is
  part of ``g_kl``.

All arithmetic is float64. Inputs are upcast to float64 as given (for the
GPU comparison the caller passes exactly the bf16 / fp32 values the GPU
reads). The only concession to memory is that ``[T, V]`` logits are formed
a block of rows at a time; rows are independent in every formula here, and
the sum over rows in ``grad_W`` is taken block by block.
"""

from __future__ import annotations

import numpy as np

IGNORE_INDEX = -100

# Rows of logits formed at once; every formula below is row-independent.
_ROW_BLOCK = 256


# ---------------------------------------------------------------------------
# helpers that restate textbook definitions
# ---------------------------------------------------------------------------

def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _logsumexp_rows(z):
    """log sum_v exp(z[t, v]) per row, with the row max factored out."""
    m = z.max(axis=1, keepdims=True)
    return (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]


def _check_problem(h, W, labels, teacher, ignore_index):
    M = len(h)
    if M < 1 or len(W) != M:
        raise ValueError("need one head per sub-model")
    T = h[0].shape[0]
    V = W[0].shape[0]
    for i in range(M):
        if h[i].ndim != 2 or W[i].ndim != 2:
            raise ValueError("h_i must be [T, d_i] and W_i must be [V, d_i]")
        if h[i].shape[0] != T or W[i].shape[0] != V or h[i].shape[1] != W[i].shape[1]:
            raise ValueError("shape mismatch between h_i and W_i")
    labels = np.asarray(labels, dtype=np.int64)
    if labels.shape != (T,):
        raise ValueError("labels must be [T]")
    bad = (labels != ignore_index) & ((labels < 0) | (labels >= V))
    if bad.any():
        raise ValueError("label out of range")
    s = M - 1 if teacher is None or teacher < 0 else int(teacher)
    if not 0 <= s < M:
        raise ValueError("teacher index out of range")
    return M, T, V, labels, s


def n_valid(labels, ignore_index=IGNORE_INDEX):
    """Number of tokens that enter the mean: labels different from ``ignore_index``."""
    return int((np.asarray(labels) != ignore_index).sum())


# ---------------------------------------------------------------------------
# loss coefficients: eq. (3), the sum over sub-models, appendix G weights
# ---------------------------------------------------------------------------

def coeffs(M, teacher=-1, alpha=0.0, tau=1.0, mode="paper", w=None):
    """Coefficients ``(g_ce, g_kl)`` of ``J = sum_i g_ce[i] CE_i + g_kl[i] KL_i``.

    ``mode="paper"``: eq. (3), ``L^m = (1 - alpha) CE_m + alpha * L_d``, for every
    sub-model with a distillation term (``m < M``); the teacher keeps its plain
    cross-entropy. The objective sums the sub-model losses, each scaled by
    ``w[m]`` (uniform weights of 1 by default; appendix G sweeps them).
    The distillation term is ``tau**2 * KL`` (temperature compensation).

    ``mode="additive"``: cross-entropy with weight 1 for every sub-model plus
    ``alpha * tau**2 * KL`` for the students (the form whose logit gradient
    reads ``softmax - onehot + alpha * (student - teacher)`` at ``tau = 1``).
    """
    s = M - 1 if teacher is None or teacher < 0 else int(teacher)
    w = np.ones(M) if w is None else _f64(w)
    g_ce = np.zeros(M)
    g_kl = np.zeros(M)
    for i in range(M):
        if i == s:
            g_ce[i] = w[i]
            g_kl[i] = 0.0
        elif mode == "paper":
            g_ce[i] = w[i] * (1.0 - alpha)
            g_kl[i] = w[i] * alpha * tau * tau
        elif mode == "additive":
            g_ce[i] = w[i]
            g_kl[i] = w[i] * alpha * tau * tau
        else:
            raise ValueError(f"unknown mode {mode!r}")
    return g_ce, g_kl


# ---------------------------------------------------------------------------
# per-row quantities for a block of rows
# ---------------------------------------------------------------------------

def _row_block_terms(h, W, labels, rows, tau, s, ignore_index):
    """Logits and per-row statistics for the given rows.

    Returns a dict with, for every sub-model ``i``:
      L[i]     logits ``h_i[rows] @ W_i^T``                 (section 2, "Modeling")
      lse1[i]  ``log sum_v exp(L_i)``                        (softmax at tau = 1)
      lset[i]  ``log sum_v exp(L_i / tau)``                  (softmax at tau)
      ce[i]    ``lse1_i - L_i[t, y_t]``, 0 on ignored rows   (next-token CE)
      kl[i]    ``sum_v q (log q - log p_i^tau)``, 0 for the teacher and on
               ignored rows                                  (eq. (2) minus H(q))
    and ``logq`` (teacher log-probabilities at tau), ``H`` (teacher entropy).
    """
    M = len(h)
    y = labels[rows]
    valid = y != ignore_index
    ysafe = np.where(valid, y, 0)
    out = {"L": [], "lse1": [], "lset": [], "ce": [], "kl": []}
    for i in range(M):
        L = _f64(h[i][rows]) @ _f64(W[i]).T
        out["L"].append(L)
        out["lse1"].append(_logsumexp_rows(L))
        out["lset"].append(_logsumexp_rows(L / tau))
        lab = L[np.arange(len(rows)), ysafe]
        out["ce"].append(np.where(valid, out["lse1"][i] - lab, 0.0))
    logq = out["L"][s] / tau - out["lset"][s][:, None]
    q = np.exp(logq)
    for i in range(M):
        if i == s:
            out["kl"].append(np.zeros(len(rows)))
            continue
        logp = out["L"][i] / tau - out["lset"][i][:, None]
        kl = (q * (logq - logp)).sum(axis=1)
        out["kl"].append(np.where(valid, kl, 0.0))
    H = -(q * logq).sum(axis=1)
    out["H"] = np.where(valid, H, 0.0)
    out["logq"] = logq
    out["valid"] = valid
    out["y"] = ysafe
    return out


def _dlogits(terms, i, s, g_ce, g_kl, tau, N):
    """Gradient of J with respect to the logits of sub-model ``i`` on a row block.

    d CE_i / d l_i   = (p_i - onehot(y)) / N                       (softmax CE)
    d KL_i / d l_i   = (p_i^tau - q) / (tau N)   with q held fixed  (stop_grad, eq. (2))
    Ignored rows contribute nothing. The teacher has no KL term.
    """
    L = terms["L"][i]
    valid = terms["valid"]
    p1 = np.exp(L - terms["lse1"][i][:, None])
    onehot = np.zeros_like(p1)
    onehot[np.arange(L.shape[0]), terms["y"]] = 1.0
    G = g_ce[i] * (p1 - onehot)
    if i != s:
        pt = np.exp(L / tau - terms["lset"][i][:, None])
        q = np.exp(terms["logq"])
        G = G + (g_kl[i] / tau) * (pt - q)
    G = G / N if N > 0 else np.zeros_like(G)
    G[~valid] = 0.0
    return G


# ---------------------------------------------------------------------------
# public API
# ---------------------------------------------------------------------------

def forward(h, W, labels, tau=1.0, teacher=-1, ignore_index=IGNORE_INDEX):
    """Losses of every sub-model.

    Returns a dict:
      ce[M], kl[M]      means over valid rows of the per-row CE and KL(q || p_i^tau)
      H                 mean teacher entropy H(q) over valid rows
      lse1[M,T], lset[M,T], ce_row[M,T], kl_row[M,T], h_row[T]
      n_valid           number of valid rows N
    With N = 0 every loss is 0.
    """
    M, T, V, labels, s = _check_problem(h, W, labels, teacher, ignore_index)
    lse1 = np.zeros((M, T))
    lset = np.zeros((M, T))
    ce_row = np.zeros((M, T))
    kl_row = np.zeros((M, T))
    h_row = np.zeros(T)
    for r0 in range(0, T, _ROW_BLOCK):
        rows = np.arange(r0, min(T, r0 + _ROW_BLOCK))
        tb = _row_block_terms(h, W, labels, rows, tau, s, ignore_index)
        for i in range(M):
            lse1[i, rows] = tb["lse1"][i]
            lset[i, rows] = tb["lset"][i]
            ce_row[i, rows] = tb["ce"][i]
            kl_row[i, rows] = tb["kl"][i]
        h_row[rows] = tb["H"]
    N = n_valid(labels, ignore_index)
    den = N if N > 0 else 1
    return {
        "ce": ce_row.sum(axis=1) / den if N > 0 else np.zeros(M),
        "kl": kl_row.sum(axis=1) / den if N > 0 else np.zeros(M),
        "H": h_row.sum() / den if N > 0 else 0.0,
        "lse1": lse1,
        "lset": lset,
        "ce_row": ce_row,
        "kl_row": kl_row,
        "h_row": h_row,
        "n_valid": N,
        "teacher": s,
    }


def backward(h, W, labels, g_ce, g_kl, tau=1.0, teacher=-1, ignore_index=IGNORE_INDEX):
    """Exact gradient of ``J = sum_i g_ce[i] CE_i + g_kl[i] KL_i`` (q under stop_grad).

    ``grad_h_i = G_i @ W_i`` and ``grad_W_i = G_i^T @ h_i`` with ``G_i`` the
    logit gradient of :func:`_dlogits` (the head is linear, section 2,
    "Modeling"). Returns ``(grad_h list, grad_W list)`` in float64.
    """
    M, T, V, labels, s = _check_problem(h, W, labels, teacher, ignore_index)
    g_ce = _f64(g_ce)
    g_kl = _f64(g_kl)
    N = n_valid(labels, ignore_index)
    grad_h = [np.zeros((T, h[i].shape[1])) for i in range(M)]
    grad_W = [np.zeros((V, h[i].shape[1])) for i in range(M)]
    for r0 in range(0, T, _ROW_BLOCK):
        rows = np.arange(r0, min(T, r0 + _ROW_BLOCK))
        tb = _row_block_terms(h, W, labels, rows, tau, s, ignore_index)
        for i in range(M):
            G = _dlogits(tb, i, s, g_ce, g_kl, tau, N)
            grad_h[i][rows] = G @ _f64(W[i])
            grad_W[i] += G.T @ _f64(h[i][rows])
    return grad_h, grad_W


def objective(h, W, labels, g_ce, g_kl, tau=1.0, teacher=-1, ignore_index=IGNORE_INDEX,
              logq_frozen=None):
    """``J = sum_i g_ce[i] CE_i + g_kl[i] KL_i``.

    With ``logq_frozen`` (teacher log-probabilities ``[T, V]`` at tau) the KL
    terms use that fixed teacher distribution: this is what ``stop_grad`` in
    eq. (2) means for a finite-difference check. Small shapes only.
    """
    M, T, V, labels, s = _check_problem(h, W, labels, teacher, ignore_index)
    rows = np.arange(T)
    tb = _row_block_terms(h, W, labels, rows, tau, s, ignore_index)
    N = n_valid(labels, ignore_index)
    if N == 0:
        return 0.0
    logq = tb["logq"] if logq_frozen is None else _f64(logq_frozen)
    q = np.exp(logq)
    J = 0.0
    for i in range(M):
        J += g_ce[i] * tb["ce"][i].sum() / N
        if i != s:
            logp = tb["L"][i] / tau - tb["lset"][i][:, None]
            kl = (q * (logq - logp)).sum(axis=1)
            J += g_kl[i] * np.where(tb["valid"], kl, 0.0).sum() / N
    return J


def teacher_logq(h, W, tau=1.0, teacher=-1):
    """Teacher log-probabilities ``log softmax(l_s / tau)`` for all rows (small shapes)."""
    M = len(h)
    s = M - 1 if teacher is None or teacher < 0 else int(teacher)
    L = _f64(h[s]) @ _f64(W[s]).T / tau
    return L - _logsumexp_rows(L)[:, None]


def per_row(h, W, labels, rows, tau=1.0, teacher=-1, ignore_index=IGNORE_INDEX):
    """Per-row statistics for a subset of rows (for sampled checks at full size).

    Returns dict with lse1[M,R], lset[M,R], ce_row[M,R], kl_row[M,R], h_row[R].
    """
    M, T, V, labels, s = _check_problem(h, W, labels, teacher, ignore_index)
    rows = np.asarray(rows, dtype=np.int64)
    tb = _row_block_terms(h, W, labels, rows, tau, s, ignore_index)
    return {
        "lse1": np.stack(tb["lse1"]),
        "lset": np.stack(tb["lset"]),
        "ce_row": np.stack(tb["ce"]),
        "kl_row": np.stack(tb["kl"]),
        "h_row": tb["H"],
    }


def grad_h_rows(h, W, labels, rows, g_ce, g_kl, tau=1.0, teacher=-1,
                ignore_index=IGNORE_INDEX):
    """Rows ``grad_h_i[rows]`` of the gradient (N is counted over all labels)."""
    M, T, V, labels, s = _check_problem(h, W, labels, teacher, ignore_index)
    rows = np.asarray(rows, dtype=np.int64)
    N = n_valid(labels, ignore_index)
    tb = _row_block_terms(h, W, labels, rows, tau, s, ignore_index)
    return [_dlogits(tb, i, s, _f64(g_ce), _f64(g_kl), tau, N) @ _f64(W[i]) for i in range(M)]


def grad_W_rows(h, W, labels, vrows, g_ce, g_kl, tau=1.0, teacher=-1,
                ignore_index=IGNORE_INDEX):
    """Rows ``grad_W_i[vrows]`` of the head gradient; needs every token's softmax."""
    M, T, V, labels, s = _check_problem(h, W, labels, teacher, ignore_index)
    vrows = np.asarray(vrows, dtype=np.int64)
    N = n_valid(labels, ignore_index)
    out = [np.zeros((len(vrows), h[i].shape[1])) for i in range(M)]
    for r0 in range(0, T, _ROW_BLOCK):
        rows = np.arange(r0, min(T, r0 + _ROW_BLOCK))
        tb = _row_block_terms(h, W, labels, rows, tau, s, ignore_index)
        for i in range(M):
            G = _dlogits(tb, i, s, _f64(g_ce), _f64(g_kl), tau, N)
            out[i] += G[:, vrows].T @ _f64(h[i][rows])
    return out


# ---------------------------------------------------------------------------
# cross-model diagnostics (section 3, "Training Dynamics and Model Agreement";
# appendix A plots the student-to-teacher direction)
# ---------------------------------------------------------------------------

def diagnostics(h, W, labels, ignore_index=IGNORE_INDEX):
    """Pairwise KL divergence and top-1 next-token agreement between sub-models.

    For every ordered pair (i, j), over the valid tokens t (label != ignore_index):
      kl[i, j]    = mean_t KL(p_i[t] || p_j[t]),  p_i = softmax(l_i) at temperature 1
      agree[i, j] = mean_t [argmax_v l_i[t] == argmax_v l_j[t]]
    argmax ties go to the lowest vocabulary index. Returns a dict with kl[M, M],
    agree[M, M], argmax[M, T] (of every token, valid or not) and n_valid; with
    no valid token kl and agree are 0.
    """
    M, T, V, labels, _ = _check_problem(h, W, labels, None, ignore_index)
    valid = labels != ignore_index
    N = int(valid.sum())
    kl_sum = np.zeros((M, M))
    agree_sum = np.zeros((M, M))
    argmax = np.zeros((M, T), dtype=np.int64)
    for r0 in range(0, T, _ROW_BLOCK):
        rows = np.arange(r0, min(T, r0 + _ROW_BLOCK))
        L = [_f64(h[i][rows]) @ _f64(W[i]).T for i in range(M)]
        logp = [Li - _logsumexp_rows(Li)[:, None] for Li in L]
        am = [np.argmax(Li, axis=1) for Li in L]  # first maximum = lowest index
        v = valid[rows]
        for i in range(M):
            argmax[i, rows] = am[i]
            p = np.exp(logp[i])
            for j in range(M):
                if i != j:
                    kl = (p * (logp[i] - logp[j])).sum(axis=1)
                    kl_sum[i, j] += kl[v].sum()
                agree_sum[i, j] += (am[i][v] == am[j][v]).sum()
    den = N if N > 0 else 1
    return {"kl": kl_sum / den if N else np.zeros((M, M)),
            "agree": agree_sum / den if N else np.zeros((M, M)),
            "argmax": argmax, "n_valid": N}
