"""Check of sampled tokens against the float64 oracle (pure numpy, no GPU).

The GPU takes the nucleus and inverse-CDF decisions in fp32 and the oracle in
fp64 on the same fp32 logits. A GPU token that differs from the oracle's is
accepted only when the oracle draws it for some (u', top_p') within EPS of
(u, top_p), with near-equal probabilities at the nucleus boundary ranked
either way, and only as many such rows as the case allows.
"""

import numpy as np

from oracle import decode as OD

EPS = 1e-5

def oracle_tokens_near(row, u, temperature, top_p):
    """Tokens the oracle draws for some (u', top_p') within EPS of (u, top_p),
    with near-equal probabilities at the nucleus boundary taken in either order.

    * The kept set changes with top_p' only where the target mass crosses a
      partial sum of the sorted probabilities, so a fine grid of top_p' values
      meets every kept set of the interval (EPS moves the target by at most
      EPS of the mass, less than one token's share on the rows tested).
    * The kernel ranks fp32 weights: tokens whose probabilities lie within
      2^-20 (relative) of the least kept one cannot be ordered reliably at that
      precision, so each swap of a kept and an unkept such token is a kept set
      too.
    * For a kept set the draw is monotone in u', so the tokens drawn over
      [u - EPS, u + EPS] are the kept tokens from the draw at u - EPS up to the
      one at u + EPS."""
    x = np.asarray(row, dtype=np.float64) / temperature
    p = np.exp(x - x.max())
    p /= p.sum()
    out = set()
    u_lo, u_hi = min(max(u - EPS, 0.0), 1.0 - 1e-12), min(max(u + EPS, 0.0), 1.0 - 1e-12)
    for pp in np.linspace(top_p - EPS, top_p + EPS, 21):
        keep = OD.filtered_probs(row, temperature, min(max(pp, 1e-9), 1.0)) > 0
        pb = p[keep].min()
        band = np.abs(p - pb) <= 2.0 ** -20 * pb
        kept_sets = [keep]
        for a in np.nonzero(band & keep)[0]:
            for b in np.nonzero(band & ~keep)[0]:
                k2 = keep.copy()
                k2[a], k2[b] = False, True
                kept_sets.append(k2)
        for k in kept_sets:
            r = np.where(k, p, 0.0)
            lo, hi = int(OD.draw(r, u_lo)), int(OD.draw(r, u_hi))
            out.update(int(v) for v in np.nonzero(r[lo:hi + 1] > 0)[0] + lo)
    return out


# Sampled rows allowed to differ from the oracle (each one still reproduced by
# it within the perturbation box), per case. The counts are deterministic for
# seeded inputs; on the GPU cases every row matches the oracle except on nearly
# flat rows over the full vocabulary (logit scale 0.01), where some 44,000 kept
# weights lie within 8 % of each other, fp32 resolves them only to ~1e-7, and
# tokens that close to the nucleus boundary can be ranked either way: 1 row of
# 24 there, allowed exactly.
FLAT_ROWS_ALLOWED = 1


def check_samples(logits, u, tokens, temperature, top_p, allowed=0):
    ref = OD.sample(logits, u, temperature, top_p)
    miss = np.nonzero(ref != tokens)[0]
    print(f"[decode] sampled tokens differing from the oracle: {len(miss)} of {len(tokens)} "
          f"(allowed {allowed})", flush=True)
    for r in miss:
        near = oracle_tokens_near(logits[r], float(u[r]), temperature, top_p)
        assert int(tokens[r]) in near, (f"row {r}: GPU token {tokens[r]}, oracle {ref[r]}, "
                                        f"oracle under perturbation {sorted(near)}")
    assert len(miss) <= allowed, f"{len(miss)} ambiguous rows, {allowed} allowed"
    return len(miss)


