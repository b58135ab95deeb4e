"""Pure-Python brute force of the Matryoshka multi-head LM loss (test infrastructure).

Tiny shapes only (a few tokens, a handful of vocabulary entries). Written
straight from the definitions with explicit loops and ``math.fsum``, sharing
no code with :mod:`oracle.mls_oracle`, whose vectorised arithmetic it pins.

Definitions (paper section 2, "Method"):
  logits        l_i[t, v] = sum_k W_i[v, k] h_i[t, k]
  softmax       p(z)_v = exp(z_v) / sum_u exp(z_u)
  cross-entropy CE_i[t] = -log p(l_i[t])_{y_t}
  eq. (2)       D_i[t] = -sum_v q_v log p(l_i[t] / tau)_v,   q = p(l_s[t] / tau)
  KL            KL_i[t] = sum_v q_v log(q_v / p(l_i[t] / tau)_v) = D_i[t] - H[t]
  entropy       H[t] = -sum_v q_v log q_v
Gradients come from the softmax Jacobian ``d log p_u / d z_v = [u == v] - p_v``
summed explicitly, not from the closed forms the vectorised oracle uses.
"""

from __future__ import annotations

import math

IGNORE = -100


def _softmax(z):
    m = max(z)
    e = [math.exp(x - m) for x in z]
    s = math.fsum(e)
    return [x / s for x in e]


def _logits(h, W):
    T = len(h)
    V = len(W)
    return [[math.fsum(W[v][k] * h[t][k] for k in range(len(h[t]))) for v in range(V)]
            for t in range(T)]


def losses(h, W, labels, tau=1.0, teacher=None):
    """Return (ce[M], kl[M], eq2[M], H, N) as Python floats (means over valid rows)."""
    M = len(h)
    s = M - 1 if teacher is None or teacher < 0 else teacher
    L = [_logits(h[i], W[i]) for i in range(M)]
    T = len(labels)
    valid = [t for t in range(T) if labels[t] != IGNORE]
    N = len(valid)
    ce = [[] for _ in range(M)]
    kl = [[] for _ in range(M)]
    d2 = [[] for _ in range(M)]
    Hs = []
    for t in valid:
        q = _softmax([x / tau for x in L[s][t]])
        Hs.append(-math.fsum(qv * math.log(qv) for qv in q if qv > 0))
        for i in range(M):
            p1 = _softmax(L[i][t])
            ce[i].append(-math.log(p1[labels[t]]))
            if i == s:
                kl[i].append(0.0)
                d2[i].append(0.0)
                continue
            pt = _softmax([x / tau for x in L[i][t]])
            kl[i].append(math.fsum(q[v] * math.log(q[v] / pt[v]) for v in range(len(q)) if q[v] > 0))
            d2[i].append(-math.fsum(q[v] * math.log(pt[v]) for v in range(len(q))))
    if N == 0:
        return [0.0] * M, [0.0] * M, [0.0] * M, 0.0, 0
    mean = lambda xs: math.fsum(xs) / N  # noqa: E731
    return ([mean(c) for c in ce], [mean(k) for k in kl], [mean(d) for d in d2],
            mean(Hs), N)


def grads(h, W, labels, g_ce, g_kl, tau=1.0, teacher=None):
    """Gradient of J = sum_i g_ce[i] CE_i + g_kl[i] KL_i with q under stop_grad.

    Returns (grad_h, grad_W) as nested lists.
    """
    M = len(h)
    s = M - 1 if teacher is None or teacher < 0 else teacher
    L = [_logits(h[i], W[i]) for i in range(M)]
    T = len(labels)
    V = len(W[0])
    N = sum(1 for y in labels if y != IGNORE)
    G = [[[0.0] * V for _ in range(T)] for _ in range(M)]
    for t in range(T):
        if labels[t] == IGNORE:
            continue
        q = _softmax([x / tau for x in L[s][t]])
        for i in range(M):
            p1 = _softmax(L[i][t])
            pt = _softmax([x / tau for x in L[i][t]])
            for v in range(V):
                # CE = -log p1[y]: d/dl_v = -([y == v] - p1[v])
                dce = -((1.0 if v == labels[t] else 0.0) - p1[v])
                # KL = sum_u q_u log q_u - sum_u q_u log pt_u, z = l / tau:
                # d/dl_v = -(1/tau) sum_u q_u ([u == v] - pt[v])
                dkl = 0.0
                if i != s:
                    dkl = -math.fsum(q[u] * ((1.0 if u == v else 0.0) - pt[v]) for u in range(V)) / tau
                G[i][t][v] = (g_ce[i] * dce + g_kl[i] * dkl) / N
    gh = [[[math.fsum(G[i][t][v] * W[i][v][k] for v in range(V)) for k in range(len(W[i][0]))]
           for t in range(T)] for i in range(M)]
    gW = [[[math.fsum(G[i][t][v] * h[i][t][k] for t in range(T)) for k in range(len(h[i][0]))]
           for v in range(V)] for i in range(M)]
    return gh, gW


def diagnostics(h, W, labels):
    """Pairwise KL(p_i || p_j) and top-1 agreement, as loops (means over valid rows)."""
    M = len(h)
    L = [_logits(h[i], W[i]) for i in range(M)]
    T = len(labels)
    valid = [t for t in range(T) if labels[t] != IGNORE]
    N = len(valid)
    kl = [[[] for _ in range(M)] for _ in range(M)]
    ag = [[0 for _ in range(M)] for _ in range(M)]
    for t in valid:
        P = [_softmax(L[i][t]) for i in range(M)]
        top = []
        for i in range(M):
            best = 0
            for v in range(1, len(L[i][t])):
                if L[i][t][v] > L[i][t][best]:
                    best = v
            top.append(best)
        for i in range(M):
            for j in range(M):
                if i != j:
                    kl[i][j].append(math.fsum(P[i][v] * math.log(P[i][v] / P[j][v])
                                              for v in range(len(P[i]))))
                ag[i][j] += 1 if top[i] == top[j] else 0
    if N == 0:
        return [[0.0] * M for _ in range(M)], [[0.0] * M for _ in range(M)]
    return ([[math.fsum(kl[i][j]) / N if i != j else 0.0 for j in range(M)] for i in range(M)],
            [[ag[i][j] / N for j in range(M)] for i in range(M)])


def junction(o, e, prev_first=True):
    """Eq. (1) as loops: each token's o rescaled to ||e|| and concatenated with e."""
    out = []
    for ot, et in zip(o, e):
        no = math.sqrt(math.fsum(x * x for x in ot))
        ne = math.sqrt(math.fsum(x * x for x in et))
        r = ne / no if no > 0 and ne > 0 else 0.0
        scaled = [x * r for x in ot]
        out.append(scaled + list(et) if prev_first else list(et) + scaled)
    return out
