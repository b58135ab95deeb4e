"""Pins of the speculative-decoding head-step oracle, and planted mistakes in it
that those pins must catch.

* brute force: the nucleus filter as pure-Python loops, and the minimal
  kept set by enumeration of every subset on tiny vocabularies;
* the inverse-CDF draw reproduces its distribution on a fine grid of uniforms;
* the speculative-sampling theorem: over the draft's distribution and
  uniform acceptance / resampling numbers, the first emitted token is
  distributed exactly as the verifier's sampling distribution;
* greedy rules, shift invariance, the top_p limits.
"""

import itertools
import math

import numpy as np
import pytest

from oracle import decode as OD


def _bf_filtered(logits, temperature, top_p):
    z = [x / temperature for x in logits]
    m = max(z)
    e = [math.exp(x - m) for x in z]
    s = math.fsum(e)
    p = [x / s for x in e]
    if top_p >= 1.0:
        return p
    idx = sorted(range(len(p)), key=lambda v: (-p[v], v))
    kept, mass = [], 0.0
    for v in idx:
        kept.append(v)
        mass = math.fsum(p[k] for k in kept)
        if mass >= top_p:
            break
    tot = math.fsum(p[k] for k in kept)
    return [p[v] / tot if v in kept else 0.0 for v in range(len(p))]


@pytest.mark.parametrize("temperature,top_p", [(1.0, 1.0), (0.4, 0.9), (0.7, 0.5), (2.0, 0.99),
                                               (0.4, 1e-6)])
def test_filter_matches_brute_force(temperature, top_p):
    rng = np.random.default_rng(1)
    for _ in range(20):
        logits = rng.standard_normal(9) * 2
        np.testing.assert_allclose(OD.filtered_probs(logits, temperature, top_p),
                                   _bf_filtered(list(logits), temperature, top_p), atol=1e-14)


def test_nucleus_is_the_smallest_set_reaching_top_p():
    rng = np.random.default_rng(2)
    for _ in range(30):
        V = 7
        logits = rng.standard_normal(V) * 1.5
        top_p = float(rng.uniform(0.05, 0.999))
        full = OD.filtered_probs(logits, 1.0, 1.0)
        kept = OD.filtered_probs(logits, 1.0, top_p) > 0
        best = None
        for n in range(1, V + 1):
            for sub in itertools.combinations(range(V), n):
                if full[list(sub)].sum() >= top_p:
                    best = n
                    break
            if best:
                break
        assert kept.sum() == best
        assert full[kept].sum() >= top_p
        # the kept tokens are the most probable ones
        assert full[kept].min() >= full[~kept].max(initial=0.0)


def test_ties_in_the_nucleus_go_to_lower_indices():
    logits = np.array([0.0, 1.0, 1.0, 1.0, -5.0])
    p = OD.filtered_probs(logits, 1.0, 0.5)  # needs two of the three tied tokens
    assert (p > 0).tolist() == [False, True, True, False, False]


def test_draw_reproduces_the_distribution():
    rng = np.random.default_rng(3)
    r = OD.filtered_probs(rng.standard_normal(11), 0.7, 0.95)
    N = 20000
    counts = np.zeros(r.size)
    for i in range(N):
        counts[OD.draw(r, (i + 0.5) / N)] += 1
    np.testing.assert_allclose(counts / N, r, atol=2.0 / N)
    assert counts[r == 0].sum() == 0


@pytest.mark.parametrize("temperature,top_p", [(1.0, 1.0), (0.4, 0.9), (0.8, 0.7)])
def test_speculative_sampling_emits_the_verifier_distribution(temperature, top_p):
    """P(first emitted token = y) = p(y) for any draft distribution q."""
    rng = np.random.default_rng(4)
    V, N = 6, 400
    for _ in range(3):
        dl = rng.standard_normal((1, 1, V)) * 1.5
        tl = rng.standard_normal((1, 2, V)) * 1.5
        p = OD.filtered_probs(tl[0, 0], temperature, top_p)
        q = OD.filtered_probs(dl[0, 0], temperature, top_p)
        dist = np.zeros(V)
        grid = (np.arange(N) + 0.5) / N
        for x in range(V):
            if q[x] == 0:
                continue
            for ua in grid:
                # u_sample only matters after a rejection: integrate it out in closed form
                n_acc, nxt = OD.verify(dl, tl, np.array([[x]]), np.array([[ua]]), np.array([0.5]),
                                       temperature, top_p)
                if n_acc[0] == 1:
                    dist[x] += q[x] / N
                else:
                    res = np.maximum(p - q, 0.0)
                    dist += q[x] / N * res / res.sum()
        np.testing.assert_allclose(dist, p, atol=2.0 / N)


def test_resampling_draws_from_the_residual():
    dl = np.array([[[3.0, 0.0, 0.0, 0.0]]])
    tl = np.array([[[0.0, 0.0, 0.0, 0.0], [0.0, 0.0, 0.0, 0.0]]])
    p = OD.filtered_probs(tl[0, 0], 1.0, 1.0)
    q = OD.filtered_probs(dl[0, 0], 1.0, 1.0)
    res = np.maximum(p - q, 0.0)
    N = 4000
    counts = np.zeros(4)
    for i in range(N):
        n_acc, nxt = OD.verify(dl, tl, np.array([[0]]), np.array([[0.999]]),
                               np.array([(i + 0.5) / N]), 1.0, 1.0)
        assert n_acc[0] == 0
        counts[nxt[0]] += 1
    np.testing.assert_allclose(counts / N, res / res.sum(), atol=2.0 / N)


def test_greedy_rules():
    rng = np.random.default_rng(5)
    B, gamma, V = 4, 5, 13
    tl = rng.standard_normal((B, gamma + 1, V))
    dl = rng.standard_normal((B, gamma, V))
    best = tl.argmax(axis=2)
    drafts = best[:, :gamma].copy()
    drafts[1, 2] = (drafts[1, 2] + 1) % V  # first mismatch at position 2
    drafts[2, 0] = (drafts[2, 0] + 3) % V  # first mismatch at position 0
    n_acc, nxt = OD.verify(dl, tl, drafts, np.zeros((B, gamma)), np.zeros(B), 0.4, 0.9,
                           greedy=True)
    assert n_acc.tolist() == [gamma, 2, 0, gamma]
    assert nxt.tolist() == [best[0, gamma], best[1, 2], best[2, 0], best[3, gamma]]
    assert OD.sample(tl[:, 0], np.zeros(B), 0.4, 0.9, greedy=True).tolist() == best[:, 0].tolist()


def test_shift_invariance_and_limits():
    rng = np.random.default_rng(6)
    logits = rng.standard_normal((5, 30)) * 2
    u = rng.uniform(size=5)
    a = OD.sample(logits, u, 0.4, 0.9)
    b = OD.sample(logits + 7.25, u, 0.4, 0.9)
    assert a.tolist() == b.tolist()
    # a tiny top_p keeps only the most probable token
    assert OD.sample(logits, u, 0.4, 1e-9).tolist() == logits.argmax(axis=1).tolist()
    # top_p = 1 is the plain temperature softmax
    z = logits[0] / 0.4
    e = np.exp(z - z.max())
    np.testing.assert_allclose(OD.filtered_probs(logits[0], 0.4, 1.0), e / e.sum(), rtol=1e-14)


# ---------------------------------------------------------------------------
# planted mistakes (patched into the oracle on the CPU only)
# ---------------------------------------------------------------------------

_orig_filtered = OD.filtered_probs
_orig_verify = OD.verify


def _mut_nucleus_drops_crossing_token(logits, temperature, top_p):
    p = _orig_filtered(logits, temperature, 1.0)
    if top_p >= 1.0:
        return p
    order = np.lexsort((np.arange(p.size), -p))
    cum = np.cumsum(p[order])
    n_keep = max(1, int(np.searchsorted(cum, top_p, side="left")))
    keep = np.zeros(p.size, dtype=bool)
    keep[order[:n_keep]] = True
    out = np.where(keep, p, 0.0)
    return out / out.sum()


def _mut_temperature_multiplies(logits, temperature, top_p):
    return _orig_filtered(np.asarray(logits) * temperature * temperature, temperature, top_p)


def _mut_residual_is_target(draft_logits, target_logits, draft_tokens, u_accept, u_sample,
                            temperature, top_p, greedy=False):
    """Resamples from p instead of max(0, p - q) after a rejection."""
    n, nxt = _orig_verify(draft_logits, target_logits, draft_tokens, u_accept, u_sample,
                          temperature, top_p, greedy)
    for b in range(len(n)):
        if n[b] < np.asarray(draft_tokens).shape[1] and not greedy:
            nxt[b] = OD.draw(OD.filtered_probs(target_logits[b][n[b]], temperature, top_p),
                             u_sample[b])
    return n, nxt


def _mut_accept_inverted(draft_logits, target_logits, draft_tokens, u_accept, u_sample,
                         temperature, top_p, greedy=False):
    """Keeps x with probability min(1, q/p)."""
    return _orig_verify(target_logits[:, :-1], np.concatenate(
        [draft_logits, target_logits[:, -1:]], axis=1), draft_tokens, u_accept, u_sample,
        temperature, top_p, greedy)


@pytest.mark.parametrize("name,filt,ver", [
    ("nucleus_drops_crossing_token", _mut_nucleus_drops_crossing_token, None),
    ("temperature_multiplies", _mut_temperature_multiplies, None),
    ("residual_is_target", None, _mut_residual_is_target),
    ("accept_inverted", None, _mut_accept_inverted),
])
def test_planted_mistake_is_caught(monkeypatch, name, filt, ver):
    if filt is not None:
        monkeypatch.setattr(OD, "filtered_probs", filt)
    if ver is not None:
        monkeypatch.setattr(OD, "verify", ver)
    checks = [lambda: test_filter_matches_brute_force(0.4, 0.9),
              test_nucleus_is_the_smallest_set_reaching_top_p,
              lambda: test_speculative_sampling_emits_the_verifier_distribution(0.4, 0.9),
              test_resampling_draws_from_the_residual,
              test_shift_invariance_and_limits]
    caught = 0
    for c in checks:
        try:
            c()
        except AssertionError:
            caught += 1
    assert caught > 0, f"mutant {name} passed every pin"


def test_empty_residual_draws_from_the_verifier():
    """Draft and verifier agree on a one-hot distribution and the drafted token
    is impossible under both: it is rejected and the next token comes from p."""
    dl = np.array([[[0.0, 40.0, 0.0, 0.0]]])
    tl = np.array([[[0.0, 40.0, 0.0, 0.0], [0.0, 0.0, 0.0, 0.0]]])
    n, x = OD.verify(dl, tl, np.array([[3]]), np.array([[0.5]]), np.array([0.3]), 0.4, 0.9)
    assert n.tolist() == [0] and x.tolist() == [1]
