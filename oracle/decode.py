"""Float64 CPU oracle of the nested speculative-decoding head step.

TEST INFRASTRUCTURE ONLY. The product path never imports this module; only
``tests/``, the smoke check and the CPU-baseline leg of ``bench.py`` do.

What is computed (paper section 2, paragraph "Speculative Decoding"; the
measured setting is section 3, "Speculative Decoding Throughput"): a smaller
sub-model ``m`` drafts ``gamma`` tokens and a larger sub-model ``m'`` verifies
them in one pass, with greedy decoding or nucleus sampling (top-p 0.9) at
temperature 0.4. The head step of either model maps hidden states to logits
with that model's LM head, ``l[t] = W o[t]``. Verification follows the
speculative sampling rule of the cited work: a drafted token ``x`` is kept
with probability ``min(1, p(x) / q(x))`` (``p`` the verifier's and ``q`` the
draft's sampling distribution at that position); at the first rejection the
next token is drawn from ``max(0, p - q)`` renormalised; if every draft token
is kept, one more token is drawn from the verifier's distribution at the
position after the drafts. Greedy verification keeps a draft token while it
equals the verifier's argmax, and emits the verifier's argmax at the first
mismatch (or after the last draft).

Readings taken where the paper does not fix the details:

* Sampling distribution: ``softmax(l / temperature)``, then the nucleus filter
  keeps the highest-probability tokens, in decreasing probability with ties in
  increasing index, up to and including the first one at which the kept mass
  reaches ``top_p``; the kept probabilities are renormalised. ``top_p = 1``
  keeps every token.
* The random numbers are inputs (uniforms in ``[0, 1)``), so any implementation
  fed the same numbers makes the same draws. A draw with uniform ``u`` from a
  distribution ``r`` over the vocabulary returns the smallest index ``v`` whose
  cumulative mass in index order ``sum_{v' <= v} r[v']`` exceeds ``u`` times the
  total mass (inverse CDF in index order; every fixed order gives the same
  distribution).
* Acceptance test: keep ``x`` when ``u * q(x) < p(x)``. This is ``u <
  p(x)/q(x)`` without a division, and it keeps tokens the draft could not have
  produced (``q(x) = 0 < p(x)``) and never keeps tokens the verifier excludes.
* Greedy argmax ties go to the lowest index.
* After a rejection, ``max(0, p - q)`` has no mass only if the rejected token
  is impossible under both distributions and the two coincide; the next token
  is then drawn from ``p``.
"""

from __future__ import annotations

import numpy as np


def head_logits(o, W):
    """``l[t, v] = sum_k o[t, k] W[v, k]`` in float64."""
    return np.asarray(o, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


def filtered_probs(logits, temperature, top_p):
    """Sampling distribution of one row: temperature softmax, then the nucleus filter."""
    z = np.asarray(logits, dtype=np.float64) / temperature
    e = np.exp(z - z.max())
    p = e / e.sum()
    if top_p >= 1.0:
        return p
    order = np.lexsort((np.arange(p.size), -p))  # decreasing p, then increasing index
    cum = np.cumsum(p[order])
    n_keep = int(np.searchsorted(cum, top_p, side="left")) + 1  # first rank reaching top_p
    n_keep = min(n_keep, p.size)
    keep = np.zeros(p.size, dtype=bool)
    keep[order[:n_keep]] = True
    out = np.where(keep, p, 0.0)
    return out / out.sum()


def draw(r, u):
    """Inverse CDF in index order: smallest v with cumsum(r)[v] > u * sum(r)."""
    c = np.cumsum(np.asarray(r, dtype=np.float64))
    v = int(np.searchsorted(c, u * c[-1], side="right"))
    return min(v, r.size - 1)


def argmax(logits):
    return int(np.argmax(np.asarray(logits)))  # first maximum = lowest index


def sample(logits, u, temperature, top_p, greedy=False):
    """Tokens of a batch of rows: ``logits [rows, V]``, ``u [rows]``."""
    logits = np.asarray(logits)
    out = np.zeros(logits.shape[0], dtype=np.int64)
    for t in range(logits.shape[0]):
        if greedy:
            out[t] = argmax(logits[t])
        else:
            out[t] = draw(filtered_probs(logits[t], temperature, top_p), u[t])
    return out


def verify(draft_logits, target_logits, draft_tokens, u_accept, u_sample, temperature, top_p,
           greedy=False):
    """Speculative verification of one batch.

    ``draft_logits [B, gamma, V]``, ``target_logits [B, gamma + 1, V]``,
    ``draft_tokens [B, gamma]``, ``u_accept [B, gamma]``, ``u_sample [B]``.
    Returns ``(n_accepted [B], next_token [B])``.
    """
    B, gamma = np.asarray(draft_tokens).shape
    n_acc = np.zeros(B, dtype=np.int64)
    nxt = np.zeros(B, dtype=np.int64)
    for b in range(B):
        k = 0
        while k < gamma:
            x = int(draft_tokens[b][k])
            if greedy:
                best = argmax(target_logits[b][k])
                if best != x:
                    nxt[b] = best
                    break
            else:
                p = filtered_probs(target_logits[b][k], temperature, top_p)
                q = filtered_probs(draft_logits[b][k], temperature, top_p)
                if not (u_accept[b][k] * q[x] < p[x]):
                    res = np.maximum(p - q, 0.0)
                    nxt[b] = draw(res if res.sum() > 0 else p, u_sample[b])
                    break
            k += 1
        n_acc[b] = k
        if k == gamma:  # every draft kept: one more token from the verifier
            if greedy:
                nxt[b] = argmax(target_logits[b][gamma])
            else:
                nxt[b] = draw(filtered_probs(target_logits[b][gamma], temperature, top_p),
                              u_sample[b])
    return n_acc, nxt
