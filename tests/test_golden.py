"""The oracles against the hand-worked fixtures under tests/golden/ (closed
forms derived by hand; each fixture states its derivation and the passage it
follows)."""

import numpy as np

from tests.golden_util import arr, ev, load
from oracle import decode as OD
from oracle import junction as OJ
from oracle import mls_oracle as oracle


def test_loss_fixture():
    g = load("loss_t1_v3.json")
    h = [arr(x) for x in g["h"]]
    W = [arr(x) for x in g["W"]]
    y = np.array(g["labels"])
    tau, alpha = ev(g["tau"]), ev(g["alpha"])
    o = oracle.forward(h, W, y, tau=tau, teacher=g["teacher"])
    ex = g["expected"]
    np.testing.assert_allclose(o["ce"], arr(ex["ce"]), rtol=1e-14)
    np.testing.assert_allclose(o["kl"], arr(ex["kl"]), rtol=1e-14, atol=1e-16)
    np.testing.assert_allclose(o["H"], ev(ex["entropy"]), rtol=1e-14)
    g_ce, g_kl = oracle.coeffs(len(h), g["teacher"], alpha=alpha, tau=tau)
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=tau, teacher=g["teacher"])
    G = arr(ex["logit_grad"])
    for i in range(len(h)):
        np.testing.assert_allclose(gW[i], G[i][:, None] * h[i][0][None, :], rtol=1e-13, atol=1e-16)
        np.testing.assert_allclose(gh[i], (G[i] @ W[i])[None, :], rtol=1e-13, atol=1e-16)


def test_nucleus_fixture():
    g = load("nucleus_and_verify_v4.json")["sample"]
    logits = arr(g["logits"])
    t, p = ev(g["temperature"]), ev(g["top_p"])
    for u, tok in g["draws"]:
        assert OD.sample(logits[None, :], np.array([ev(u)]), t, p)[0] == tok
    assert OD.sample(logits[None, :], np.zeros(1), t, p, greedy=True)[0] == g["greedy"]


def test_verify_fixture():
    g = load("nucleus_and_verify_v4.json")["verify"]
    dl = arr(g["draft_logits"])[None, None, :]
    tl = arr(g["target_logits"])[None, :, :]
    t, p = ev(g["temperature"]), ev(g["top_p"])
    for c in g["cases"]:
        n, x = OD.verify(dl, tl, np.array([[g["draft_token"]]]), np.array([[ev(c["u_accept"])]]),
                         np.array([ev(c["u_sample"])]), t, p)
        assert (int(n[0]), int(x[0])) == (c["n_accepted"], c["next_token"]), c


def test_junction_fixture():
    g = load("junction_3_4.json")
    o, e, gx = arr(g["o"]), arr(g["e"]), arr(g["g_x"])
    ex = g["expected"]
    np.testing.assert_allclose(OJ.forward(o, e), arr(ex["x"]), rtol=1e-15, atol=1e-16)
    g_o, g_e = OJ.backward(o, e, gx)
    np.testing.assert_allclose(g_o, arr(ex["g_o"]), rtol=1e-14, atol=1e-16)
    np.testing.assert_allclose(g_e, arr(ex["g_e"]), rtol=1e-14, atol=1e-16)


def test_evaluator_accepts_only_closed_forms():
    import pytest
    assert ev("ln(3)/2 + ln(3/4)/4") == np.log(3) / 2 + np.log(0.75) / 4
    for bad in ("__import__('os')", "exp(1)", "[1]", "1 ** 2"):
        with pytest.raises(ValueError):
            ev(bad)
