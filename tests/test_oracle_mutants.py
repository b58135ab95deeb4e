"""Planted mistakes in the CPU oracle must be caught by its pins.

Each mutant patches one step of :mod:`oracle.mls_oracle` on the CPU (a dropped
factor, a wrong sign, a wrong index, a wrong normaliser) and the test checks
that the brute-force pin or the finite-difference pin rejects it.
"""

import numpy as np
import pytest

import oracle
from oracle import bruteforce
from oracle import mls_oracle as om

_orig_dlogits = om._dlogits
_orig_terms = om._row_block_terms


def _mut_dlogits_no_inv_tau(terms, i, s, g_ce, g_kl, tau, N):
    return _orig_dlogits(terms, i, s, g_ce, np.asarray(g_kl) * tau, tau, N)


def _mut_dlogits_q_sign(terms, i, s, g_ce, g_kl, tau, N):
    """Uses (p^tau + q) in place of (p^tau - q)."""
    G = _orig_dlogits(terms, i, s, g_ce, g_kl, tau, N)
    if i != s and N > 0:
        extra = 2.0 * (g_kl[i] / tau) * np.exp(terms["logq"]) / N
        extra[~terms["valid"]] = 0.0
        G = G + extra
    return G


def _mut_dlogits_count_all_rows(terms, i, s, g_ce, g_kl, tau, N):
    return _orig_dlogits(terms, i, s, g_ce, g_kl, tau, len(terms["valid"]))


def _mut_terms_lset_is_lse1(h, W, labels, rows, tau, s, ignore_index):
    out = _orig_terms(h, W, labels, rows, tau, s, ignore_index)
    out["lset"] = list(out["lse1"])
    return out


def _mut_terms_label_shift(h, W, labels, rows, tau, s, ignore_index):
    V = W[0].shape[0]
    lab = np.where(labels == ignore_index, labels, (labels + 1) % V)
    return _orig_terms(h, W, lab, rows, tau, s, ignore_index)


def _mut_terms_teacher_index(h, W, labels, rows, tau, s, ignore_index):
    return _orig_terms(h, W, labels, rows, tau, 0 if s != 0 else 1, ignore_index)


MUTANTS = {
    "kl_grad_missing_1_over_tau": ("_dlogits", _mut_dlogits_no_inv_tau),
    "q_term_sign": ("_dlogits", _mut_dlogits_q_sign),
    "mean_over_all_rows": ("_dlogits", _mut_dlogits_count_all_rows),
    "tau_softmax_uses_tau1_lse": ("_row_block_terms", _mut_terms_lset_is_lse1),
    "label_off_by_one": ("_row_block_terms", _mut_terms_label_shift),
    "wrong_teacher": ("_row_block_terms", _mut_terms_teacher_index),
}


def _pins_pass():
    """Brute-force comparison of losses and gradients on one small case."""
    M, T, dims, V, tau = 3, 4, (2, 3, 2), 6, 1.7
    r = np.random.default_rng(101)
    h = [r.normal(size=(T, d)) for d in dims]
    W = [r.normal(scale=0.8, size=(V, d)) for d in dims]
    y = r.integers(0, V, size=T)
    y[2] = oracle.IGNORE_INDEX
    g_ce = np.array([0.6, 0.9, 1.0])
    g_kl = np.array([1.3, 0.7, 0.0])
    try:
        o = oracle.forward(h, W, y, tau=tau)
        gh, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=tau)
    except Exception:
        return False
    tl = lambda a: [x.tolist() for x in a]  # noqa: E731
    ce, kl, _, H, N = bruteforce.losses(tl(h), tl(W), y.tolist(), tau, -1)
    bh, bW = bruteforce.grads(tl(h), tl(W), y.tolist(), g_ce.tolist(), g_kl.tolist(), tau, -1)
    ok = np.allclose(o["ce"], ce, rtol=1e-10) and np.allclose(o["kl"], kl, rtol=1e-10)
    for i in range(M):
        ok = ok and np.allclose(gh[i], bh[i], rtol=1e-9, atol=1e-13)
        ok = ok and np.allclose(gW[i], bW[i], rtol=1e-9, atol=1e-13)
    return bool(ok)


def test_unmutated_oracle_passes():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(om, attr, fn)
    assert not _pins_pass(), f"planted mistake {name!r} was not caught"
