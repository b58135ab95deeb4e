"""The HIP path against the hand-worked fixtures under tests/golden/ (closed
forms derived by hand). Inputs are zero-padded to the path's minimum widths
(fp32 widths are multiples of 4, junction widths multiples of 8), which
leaves the logits and norms unchanged."""

import numpy as np
import pytest
import torch

from paper_2608_09703_amd import api as D
from tests.golden_util import arr, ev, load
from tests.gpu_helpers import run_gpu

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _t(x, dtype=torch.float32):
    return torch.tensor(np.asarray(x), dtype=dtype, device=DEV)


def test_loss_fixture_on_gpu():
    print("[golden] loss T=1 V=3", flush=True)
    g = load("loss_t1_v3.json")
    pad = 4
    h, W = [], []
    for hi, Wi in zip(g["h"], g["W"]):
        a, b = arr(hi), arr(Wi)
        h.append(_t(np.pad(a, ((0, 0), (0, pad - a.shape[1])))))
        W.append(_t(np.pad(b, ((0, 0), (0, pad - b.shape[1])))))
    y = torch.tensor(g["labels"], dtype=torch.int64, device=DEV)
    out = run_gpu(h, W, y, tau=ev(g["tau"]), teacher=g["teacher"], alpha=ev(g["alpha"]))
    ex = g["expected"]
    np.testing.assert_allclose(out["ce"], arr(ex["ce"]), rtol=1e-6)
    np.testing.assert_allclose(out["kl"], arr(ex["kl"]), rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(out["H"], ev(ex["entropy"]), rtol=1e-6)
    G = arr(ex["logit_grad"])
    for i in range(2):
        Wn = W[i].cpu().numpy().astype(np.float64)
        np.testing.assert_allclose(out["grad_W"][i][:, 0], G[i], rtol=1e-5, atol=1e-6)
        np.testing.assert_allclose(out["grad_W"][i][:, 1:], 0.0, atol=0)
        np.testing.assert_allclose(out["grad_h"][i][0], G[i] @ Wn, rtol=1e-5, atol=1e-6)


def test_nucleus_fixture_on_gpu():
    print("[golden] nucleus V=4", flush=True)
    g = load("nucleus_and_verify_v4.json")["sample"]
    n = len(g["draws"])
    logits = _t(np.tile(arr(g["logits"]), (n, 1)))
    u = _t([ev(d[0]) for d in g["draws"]])
    tok = D.sample(logits, u, temperature=ev(g["temperature"]), top_p=ev(g["top_p"]))
    assert tok.cpu().tolist() == [d[1] for d in g["draws"]]
    assert D.sample(logits, None, greedy=True).cpu().tolist() == [g["greedy"]] * n


def test_verify_fixture_on_gpu():
    print("[golden] verify V=4 gamma=1", flush=True)
    g = load("nucleus_and_verify_v4.json")["verify"]
    cases = g["cases"]
    B = len(cases)
    dl = _t(np.tile(arr(g["draft_logits"]), (1, B, 1)))           # [gamma=1][B][V]
    tl = _t(np.tile(arr(g["target_logits"])[None], (B, 1, 1)))   # [B][gamma + 1][V]
    drafts = torch.full((1, B), g["draft_token"], dtype=torch.int32, device=DEV)
    ua = _t([[ev(c["u_accept"]) for c in cases]])
    us = _t([ev(c["u_sample"]) for c in cases])
    n, x = D.spec_verify(dl, tl, drafts, ua, us, temperature=ev(g["temperature"]),
                         top_p=ev(g["top_p"]))
    assert n.cpu().tolist() == [c["n_accepted"] for c in cases]
    assert x.cpu().tolist() == [c["next_token"] for c in cases]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_junction_fixture_on_gpu(dtype):
    print(f"[golden] junction {dtype}", flush=True)
    g = load("junction_3_4.json")
    ex = g["expected"]
    w = 8
    o, e = arr(g["o"]), arr(g["e"])
    dp, df = o.shape[1], e.shape[1]
    op = np.pad(o, ((0, 0), (0, w - dp)))
    ep = np.pad(e, ((0, 0), (0, w - df)))
    gx = arr(g["g_x"])
    gxp = np.concatenate([np.pad(gx[:, :dp], ((0, 0), (0, w - dp))),
                          np.pad(gx[:, dp:], ((0, 0), (0, w - df)))], axis=1)
    xr = arr(ex["x"])
    x_exp = np.concatenate([np.pad(xr[:, :dp], ((0, 0), (0, w - dp))),
                            np.pad(xr[:, dp:], ((0, 0), (0, w - df)))], axis=1)
    x = D.junction_forward(_t(op, dtype), _t(ep, dtype)).float().cpu().numpy()
    tol = dict(rtol=2.0 ** -8, atol=1e-7) if dtype == torch.bfloat16 else dict(rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(x, x_exp, **tol)
    g_o, g_e = D.junction_backward(_t(op, dtype), _t(ep, dtype), _t(gxp, torch.float32))
    np.testing.assert_allclose(g_o.cpu().numpy()[:, :dp], arr(ex["g_o"]), rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(g_o.cpu().numpy()[:, dp:], 0.0, atol=0)
    np.testing.assert_allclose(g_e.cpu().numpy()[:, :df], arr(ex["g_e"]), rtol=1e-6, atol=1e-7)
