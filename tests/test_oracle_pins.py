"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

The paper prints no worked numerical example of its losses, so the oracle
is pinned by: a pure-Python brute force of the definitions, central finite
differences of the objective (teacher distribution frozen, as ``stop_grad``
in eq. (2) requires), closed forms (uniform logits, V = 2, a hand-worked
three-word example, the tau = 1 logit gradient), invariants (KL = 0 for a
student equal to its teacher, zero row sums of the logit gradient, shift
invariance, ignored rows) and an independent library routine (float64
PyTorch cross-entropy / KL divergence and autograd on the CPU).
"""

import math

import numpy as np
import pytest

import oracle
from oracle import bruteforce

RNG = np.random.default_rng


def _problem(M, T, dims, V, seed, w_std=0.7, ignore=()):
    r = RNG(seed)
    h = [r.normal(size=(T, d)) for d in dims]
    W = [r.normal(scale=w_std, size=(V, d)) for d in dims]
    y = r.integers(0, V, size=T)
    for t in ignore:
        y[t] = oracle.IGNORE_INDEX
    return h, W, y


def _tolist(a):
    return [np.asarray(x).tolist() for x in a]


# ----------------------------------------------------------------------------
# brute force (definitions as loops with math.fsum)
# ----------------------------------------------------------------------------

BF_CASES = [
    # M, T, dims, V, tau, teacher, ignore
    (1, 3, (2,), 5, 1.0, -1, ()),
    (2, 4, (2, 3), 7, 1.0, -1, (1,)),
    (3, 4, (1, 2, 3), 6, 0.7, -1, ()),
    (3, 3, (3, 2, 3), 5, 2.0, 0, (0,)),
    (2, 4, (3, 3), 2, 1.5, -1, (2, 3)),
]


@pytest.mark.parametrize("case", BF_CASES)
def test_bruteforce_losses(case):
    M, T, dims, V, tau, teacher, ign = case
    h, W, y = _problem(M, T, dims, V, seed=11 + T * V, ignore=ign)
    o = oracle.forward(h, W, y, tau=tau, teacher=teacher)
    ce, kl, eq2, H, N = bruteforce.losses(_tolist(h), _tolist(W), y.tolist(), tau, teacher)
    assert o["n_valid"] == N
    np.testing.assert_allclose(o["ce"], ce, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(o["kl"], kl, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(o["H"], H, rtol=1e-12, atol=1e-13)
    s = M - 1 if teacher < 0 else teacher
    # eq. (2) (teacher-weighted cross-entropy) = KL + H for every student
    for i in range(M):
        if i != s:
            np.testing.assert_allclose(o["kl"][i] + o["H"], eq2[i], rtol=1e-12)


@pytest.mark.parametrize("case", BF_CASES)
def test_bruteforce_grads(case):
    M, T, dims, V, tau, teacher, ign = case
    h, W, y = _problem(M, T, dims, V, seed=23 + T * V, ignore=ign)
    r = RNG(5)
    g_ce = r.uniform(0.2, 1.5, size=M)
    g_kl = r.uniform(0.2, 1.5, size=M)
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=tau, teacher=teacher)
    bh, bW = bruteforce.grads(_tolist(h), _tolist(W), y.tolist(), g_ce.tolist(), g_kl.tolist(),
                              tau, teacher)
    for i in range(M):
        np.testing.assert_allclose(gh[i], bh[i], rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(gW[i], bW[i], rtol=1e-11, atol=1e-14)


# ----------------------------------------------------------------------------
# finite differences with the teacher frozen (stop_grad of eq. (2))
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("tau,teacher", [(1.0, -1), (2.0, -1), (0.5, 1)])
def test_finite_differences(tau, teacher):
    M, T, dims, V = 3, 5, (3, 4, 5), 9
    h, W, y = _problem(M, T, dims, V, seed=7, ignore=(3,))
    g_ce, g_kl = oracle.coeffs(M, teacher, alpha=0.4, tau=tau, mode="paper")
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=tau, teacher=teacher)
    logq = oracle.teacher_logq(h, W, tau=tau, teacher=teacher)
    eps = 1e-5

    def J(hh, WW):
        return oracle.objective(hh, WW, y, g_ce, g_kl, tau=tau, teacher=teacher, logq_frozen=logq)

    for i in range(M):
        for arr, grad in ((h, gh), (W, gW)):
            num = np.zeros_like(arr[i])
            for idx in np.ndindex(arr[i].shape):
                old = arr[i][idx]
                arr[i][idx] = old + eps
                jp = J(h, W)
                arr[i][idx] = old - eps
                jm = J(h, W)
                arr[i][idx] = old
                num[idx] = (jp - jm) / (2 * eps)
            err = np.abs(num - grad[i]).max() / max(np.abs(grad[i]).max(), 1e-12)
            assert err < 1e-7, (i, err)


def test_teacher_gets_no_distillation_gradient():
    """With only KL coefficients, the teacher's gradients are exactly zero (stop_grad)."""
    M, T, dims, V = 3, 4, (2, 3, 4), 6
    h, W, y = _problem(M, T, dims, V, seed=3)
    g_ce = np.zeros(M)
    g_kl = np.ones(M)
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl)
    assert np.all(gh[M - 1] == 0) and np.all(gW[M - 1] == 0)
    assert np.abs(gh[0]).max() > 0


# ----------------------------------------------------------------------------
# closed forms
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("V", [2, 7, 4096, 50304])
def test_uniform_logits(V):
    """W_i = 0: every logit equal, CE = ln V exactly, KL = 0, G = g_ce (1/V - e_y) / N."""
    M, T, dims = 2, 3, (4, 5)
    r = RNG(1)
    h = [r.normal(size=(T, d)) for d in dims]
    W = [np.zeros((V, d)) for d in dims]
    y = r.integers(0, V, size=T)
    o = oracle.forward(h, W, y, tau=1.3)
    np.testing.assert_allclose(o["ce"], math.log(V), rtol=1e-14)
    np.testing.assert_allclose(o["kl"], 0.0, atol=1e-14)
    np.testing.assert_allclose(o["H"], math.log(V), rtol=1e-14)
    if V <= 4096:
        g_ce, g_kl = np.array([0.7, 1.0]), np.array([0.3, 0.0])
        _, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=1.3)
        for i in range(M):
            G = np.full((T, V), 1.0 / V)
            G[np.arange(T), y] -= 1.0
            G *= g_ce[i] / T
            np.testing.assert_allclose(gW[i], G.T @ h[i], rtol=1e-12, atol=1e-15)


def test_hand_worked_three_word_example():
    """T = 1, V = 3, d = 1, label 1.

    Student logits (0, ln 2, ln 3): p = (1/6, 1/3, 1/2).
    Teacher logits (ln 2, 0, 0):    q = (1/2, 1/4, 1/4).
    CE_student = ln 3, CE_teacher = ln 4,
    KL(q || p) = 1/2 ln 3 + 1/4 ln(3/4) + 1/4 ln(1/2), H(q) = 3/2 ln 2,
    eq. (2) value -sum q ln p = 3/4 ln 2 + 3/4 ln 3 = KL + H.
    tau = 1, alpha = 0.3, paper mode: student logit gradient p - 0.7 e_y - 0.3 q,
    teacher logit gradient p_T - e_y with p_T = q.
    """
    ln2, ln3 = math.log(2), math.log(3)
    h = [np.array([[1.0]]), np.array([[1.0]])]
    W = [np.array([[0.0], [ln2], [ln3]]), np.array([[ln2], [0.0], [0.0]])]
    y = np.array([1])
    o = oracle.forward(h, W, y)
    assert o["ce"][0] == pytest.approx(ln3, rel=1e-15)
    assert o["ce"][1] == pytest.approx(math.log(4), rel=1e-15)
    kl = 0.5 * ln3 + 0.25 * math.log(0.75) + 0.25 * math.log(0.5)
    assert o["kl"][0] == pytest.approx(kl, rel=1e-14)
    assert o["kl"][1] == 0.0
    assert o["H"] == pytest.approx(1.5 * ln2, rel=1e-15)
    assert o["kl"][0] + o["H"] == pytest.approx(0.75 * (ln2 + ln3), rel=1e-14)
    g_ce, g_kl = oracle.coeffs(2, -1, alpha=0.3, tau=1.0)
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl)
    Gs = np.array([1 / 6 - 0.15, 1 / 3 - 0.7 - 0.075, 0.5 - 0.075])
    Gt = np.array([0.5, 0.25 - 1.0, 0.25])
    np.testing.assert_allclose(gW[0][:, 0], Gs, rtol=1e-14, atol=1e-16)
    np.testing.assert_allclose(gW[1][:, 0], Gt, rtol=1e-14, atol=1e-16)
    assert gh[0][0, 0] == pytest.approx(Gs[1] * ln2 + Gs[2] * ln3, rel=1e-14)
    assert gh[1][0, 0] == pytest.approx(Gt[0] * ln2, rel=1e-14)


def test_binary_vocab_closed_form():
    """V = 2: CE = softplus(l_other - l_y); KL is the Bernoulli divergence."""
    M, T, dims, V = 2, 6, (3, 4), 2
    h, W, y = _problem(M, T, dims, V, seed=9)
    tau = 1.7
    o = oracle.forward(h, W, y, tau=tau)
    L = [h[i] @ W[i].T for i in range(M)]
    for i in range(M):
        other = 1 - y
        z = L[i][np.arange(T), other] - L[i][np.arange(T), y]
        np.testing.assert_allclose(o["ce_row"][i], np.logaddexp(0.0, z), rtol=1e-13)
    sig = lambda x: 1.0 / (1.0 + np.exp(-x))  # noqa: E731
    q1 = sig((L[1][:, 1] - L[1][:, 0]) / tau)
    p1 = sig((L[0][:, 1] - L[0][:, 0]) / tau)
    kl = q1 * np.log(q1 / p1) + (1 - q1) * np.log((1 - q1) / (1 - p1))
    np.testing.assert_allclose(o["kl_row"][0], kl, rtol=1e-12)


def test_tau1_paper_mode_logit_gradient():
    """tau = 1, paper mode: student logit gradient = (p - (1 - a) e_y - a q) / N."""
    from scipy.special import softmax

    M, T, dims, V = 2, 5, (3, 6), 11
    h, W, y = _problem(M, T, dims, V, seed=13, ignore=(2,))
    a = 0.35
    g_ce, g_kl = oracle.coeffs(M, -1, alpha=a, tau=1.0, mode="paper")
    _, gW = oracle.backward(h, W, y, g_ce, g_kl)
    p = softmax(h[0] @ W[0].T, axis=1)
    q = softmax(h[1] @ W[1].T, axis=1)
    e = np.zeros((T, V))
    e[np.arange(T), np.where(y >= 0, y, 0)] = 1.0
    N = int((y >= 0).sum())
    G = (p - (1 - a) * e - a * q) / N
    G[y < 0] = 0.0
    np.testing.assert_allclose(gW[0], G.T @ h[0], rtol=1e-12, atol=1e-15)


# ----------------------------------------------------------------------------
# invariants
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("tau", [1.0, 2.0, 0.6])
def test_identical_student_has_zero_kl(tau):
    M, T, d, V = 3, 6, 5, 13
    h, W, y = _problem(M, T, (d, d, d), V, seed=17)
    h[0] = h[2].copy()
    W[0] = W[2].copy()
    o = oracle.forward(h, W, y, tau=tau)
    assert abs(o["kl"][0]) < 1e-14
    assert o["kl"][1] > 1e-3
    g_ce = np.zeros(M)
    g_kl = np.ones(M)
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=tau)
    assert np.abs(gh[0]).max() < 1e-14 and np.abs(gW[0]).max() < 1e-14


def test_logit_gradient_rows_sum_to_zero():
    """Every row of G_i sums to zero, so sum_v grad_W_i[v, :] = 0."""
    M, T, dims, V = 3, 7, (4, 5, 6), 19
    h, W, y = _problem(M, T, dims, V, seed=19, ignore=(0, 4))
    g_ce, g_kl = oracle.coeffs(M, -1, alpha=0.6, tau=1.4, mode="additive")
    _, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=1.4)
    for i in range(M):
        assert np.abs(gW[i].sum(axis=0)).max() < 1e-14


def test_ranges():
    M, T, dims, V = 3, 8, (4, 5, 6), 17
    for tau in (0.5, 1.0, 3.0):
        h, W, y = _problem(M, T, dims, V, seed=int(tau * 10), w_std=2.0)
        o = oracle.forward(h, W, y, tau=tau)
        assert np.all(o["ce"] >= 0) and np.all(o["kl"] >= 0)
        assert 0 <= o["H"] <= math.log(V) + 1e-12


def test_shift_invariance():
    """A constant feature with a vocabulary-constant head column shifts every logit."""
    M, T, dims, V = 2, 5, (3, 4), 9
    h, W, y = _problem(M, T, dims, V, seed=29)
    h2 = [np.concatenate([x, np.ones((T, 1))], axis=1) for x in h]
    W2 = [np.concatenate([w, np.full((V, 1), 2.5)], axis=1) for w in W]
    g_ce, g_kl = oracle.coeffs(M, -1, alpha=0.5, tau=1.3)
    o1 = oracle.forward(h, W, y, tau=1.3)
    o2 = oracle.forward(h2, W2, y, tau=1.3)
    for k in ("ce", "kl"):
        np.testing.assert_allclose(o1[k], o2[k], rtol=1e-12)
    gh1, gW1 = oracle.backward(h, W, y, g_ce, g_kl, tau=1.3)
    gh2, gW2 = oracle.backward(h2, W2, y, g_ce, g_kl, tau=1.3)
    for i in range(M):
        np.testing.assert_allclose(gh2[i][:, :-1], gh1[i], rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(gW2[i][:, :-1], gW1[i], rtol=1e-11, atol=1e-14)
        assert np.abs(gh2[i][:, -1]).max() < 1e-14


def test_ignored_rows():
    """Ignored rows get zero grad_h, do not touch grad_W, and are not counted in N."""
    M, T, dims, V = 2, 6, (3, 4), 8
    h, W, y = _problem(M, T, dims, V, seed=31, ignore=(1, 4))
    g_ce, g_kl = oracle.coeffs(M, -1, alpha=0.5, tau=1.0)
    o = oracle.forward(h, W, y)
    assert o["n_valid"] == 4
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl)
    for i in range(M):
        assert np.all(gh[i][[1, 4]] == 0)
    keep = [0, 2, 3, 5]
    o2 = oracle.forward([x[keep] for x in h], W, y[keep])
    np.testing.assert_allclose(o["ce"], o2["ce"], rtol=1e-13)
    np.testing.assert_allclose(o["kl"], o2["kl"], rtol=1e-13)
    _, gW2 = oracle.backward([x[keep] for x in h], W, y[keep], g_ce, g_kl)
    for i in range(M):
        np.testing.assert_allclose(gW[i], gW2[i], rtol=1e-12, atol=1e-15)


def test_all_rows_ignored_gives_zero():
    M, T, dims, V = 2, 3, (2, 3), 5
    h, W, y = _problem(M, T, dims, V, seed=37, ignore=(0, 1, 2))
    o = oracle.forward(h, W, y)
    assert o["n_valid"] == 0
    assert np.all(o["ce"] == 0) and np.all(o["kl"] == 0) and o["H"] == 0
    gh, gW = oracle.backward(h, W, y, np.ones(M), np.ones(M))
    assert all(np.all(x == 0) for x in gh + gW)


def test_label_out_of_range_raises():
    h, W, y = _problem(2, 3, (2, 2), 4, seed=41)
    y[1] = 4
    with pytest.raises(ValueError):
        oracle.forward(h, W, y)


def test_coefficients():
    """eq. (3) with the sum over sub-models; tau^2 on the distillation term."""
    g_ce, g_kl = oracle.coeffs(3, -1, alpha=0.3, tau=2.0, mode="paper", w=[1, 2, 3])
    np.testing.assert_allclose(g_ce, [0.7, 1.4, 3.0])
    np.testing.assert_allclose(g_kl, [1.2, 2.4, 0.0])
    g_ce, g_kl = oracle.coeffs(3, 0, alpha=0.5, tau=1.0, mode="additive")
    np.testing.assert_allclose(g_ce, [1, 1, 1])
    np.testing.assert_allclose(g_kl, [0, 0.5, 0.5])


# ----------------------------------------------------------------------------
# independent library routine: float64 PyTorch on the CPU
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("tau,teacher", [(1.0, -1), (2.0, -1), (0.8, 0)])
def test_torch_cpu_float64_crosscheck(tau, teacher):
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    M, T, dims, V = 3, 12, (8, 16, 24), 37
    h, W, y = _problem(M, T, dims, V, seed=43, ignore=(2, 7))
    s = M - 1 if teacher < 0 else teacher
    g_ce, g_kl = oracle.coeffs(M, teacher, alpha=0.3, tau=tau, mode="paper", w=[0.5, 1.0, 2.0])
    o = oracle.forward(h, W, y, tau=tau, teacher=teacher)
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=tau, teacher=teacher)

    th = [torch.tensor(x, requires_grad=True) for x in h]
    tW = [torch.tensor(x, requires_grad=True) for x in W]
    ty = torch.tensor(y)
    valid = ty != -100
    logits = [th[i] @ tW[i].T for i in range(M)]
    logq = F.log_softmax(logits[s].detach() / tau, dim=1)
    J = 0.0
    for i in range(M):
        ce = F.cross_entropy(logits[i], ty, ignore_index=-100, reduction="mean")
        assert ce.item() == pytest.approx(o["ce"][i], rel=1e-12)
        J = J + g_ce[i] * ce
        if i != s:
            lp = F.log_softmax(logits[i][valid] / tau, dim=1)
            kl = F.kl_div(lp, logq[valid], log_target=True, reduction="sum") / int(valid.sum())
            assert kl.item() == pytest.approx(o["kl"][i], rel=1e-12)
            J = J + g_kl[i] * kl
    J.backward()
    for i in range(M):
        np.testing.assert_allclose(th[i].grad.numpy(), gh[i], rtol=1e-10, atol=1e-15)
        np.testing.assert_allclose(tW[i].grad.numpy(), gW[i], rtol=1e-10, atol=1e-15)


def test_sampled_row_helpers_agree_with_full():
    M, T, dims, V = 3, 9, (3, 4, 5), 10
    h, W, y = _problem(M, T, dims, V, seed=47, ignore=(5,))
    g_ce, g_kl = oracle.coeffs(M, -1, alpha=0.5, tau=1.5)
    o = oracle.forward(h, W, y, tau=1.5)
    gh, gW = oracle.backward(h, W, y, g_ce, g_kl, tau=1.5)
    rows = [0, 5, 8]
    pr = oracle.per_row(h, W, y, rows, tau=1.5)
    for k in ("lse1", "lset", "ce_row", "kl_row"):
        np.testing.assert_allclose(pr[k], o[k][:, rows], rtol=1e-13)
    ghr = oracle.grad_h_rows(h, W, y, rows, g_ce, g_kl, tau=1.5)
    gWr = oracle.grad_W_rows(h, W, y, [1, 9], g_ce, g_kl, tau=1.5)
    for i in range(M):
        np.testing.assert_allclose(ghr[i], gh[i][rows], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(gWr[i], gW[i][[1, 9]], rtol=1e-12, atol=1e-15)


# ----------------------------------------------------------------------------
# cross-model diagnostics: pairwise KL and top-1 agreement
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [61, 62])
def test_diagnostics_bruteforce(seed):
    M, T, dims, V = 3, 5, (2, 3, 2), 7
    h, W, y = _problem(M, T, dims, V, seed=seed, ignore=(1,))
    o = oracle.diagnostics(h, W, y)
    kl, ag = bruteforce.diagnostics(_tolist(h), _tolist(W), y.tolist())
    np.testing.assert_allclose(o["kl"], kl, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(o["agree"], ag, rtol=0, atol=0)


def test_diagnostics_invariants():
    M, T, dims, V = 3, 40, (4, 5, 4), 23
    h, W, y = _problem(M, T, dims, V, seed=63, ignore=(3, 9))
    h[2] = h[0].copy()
    W[2] = W[0].copy()
    o = oracle.diagnostics(h, W, y)
    assert np.all(np.diag(o["kl"]) == 0) and np.all(np.diag(o["agree"]) == 1)
    assert np.all(o["kl"] >= -1e-15)
    assert abs(o["kl"][0, 2]) < 1e-14 and abs(o["kl"][2, 0]) < 1e-14 and o["agree"][0, 2] == 1
    assert o["kl"][0, 1] > 1e-3 and o["kl"][0, 1] != pytest.approx(o["kl"][1, 0], rel=1e-6)
    # the training loss's KL(q || p_i) at tau = 1 is the teacher-to-student entry
    f = oracle.forward(h, W, y, tau=1.0)
    np.testing.assert_allclose(f["kl"][:2], o["kl"][2, :2], rtol=1e-12, atol=1e-15)


def test_diagnostics_argmax_ties_to_lowest_index():
    """Tied maxima: every head maps to the same logits for vocabulary rows 2 and 5."""
    h = [np.array([[1.0], [2.0]]), np.array([[1.0], [-1.0]])]
    W = [np.array([[0.0], [1.0], [3.0], [2.0], [0.5], [3.0]]),
         np.array([[4.0], [0.0], [1.0], [4.0], [-1.0], [0.0]])]
    y = np.array([0, 1])
    o = oracle.diagnostics(h, W, y)
    assert o["argmax"][0].tolist() == [2, 2]
    assert o["argmax"][1].tolist() == [0, 4]
    assert o["agree"][0, 1] == 0.0


def test_diagnostics_torch_crosscheck():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    M, T, dims, V = 3, 16, (8, 12, 16), 29
    h, W, y = _problem(M, T, dims, V, seed=64, ignore=(5,))
    o = oracle.diagnostics(h, W, y)
    v = torch.tensor(y != -100)
    L = [torch.tensor(h[i]) @ torch.tensor(W[i]).T for i in range(M)]
    lp = [F.log_softmax(x, dim=1)[v] for x in L]
    for i in range(M):
        for j in range(M):
            if i != j:
                ref = F.kl_div(lp[j], lp[i], log_target=True, reduction="sum").item() / int(v.sum())
                assert o["kl"][i, j] == pytest.approx(ref, rel=1e-12)
            agree = (L[i].argmax(dim=1)[v] == L[j].argmax(dim=1)[v]).double().mean().item()
            assert o["agree"][i, j] == pytest.approx(agree, abs=1e-15)
