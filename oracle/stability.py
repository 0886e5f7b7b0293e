"""Drop-set stability signals -- TEST INFRASTRUCTURE ONLY.

Paper section 3.4, UCS operators (3) diffusion-head cache reuse and (4)
denoising-step early exit. For one sequence at two timesteps t and t_ref the
router's drop set D_t is the set of routable tokens it does not retain.

  J(t, t_ref)   = |D_t n D_ref| / |D_t u D_ref|                    (Eq. 10)
  RDA(t, t_ref) = (J - J_rand) / (1 - J_rand)                       (Eq. 11)

J_rand is the Jaccard similarity expected when the same numbers of tokens are
dropped at random. Readings taken here (the paper does not spell them out):
  * the universe is the sequence's routable tokens (always-kept tokens are
    never dropped, so they are in neither set);
  * J_rand is the exact expectation of J for two independent, uniformly random
    subsets A, B of that universe with |A| = |D_t|, |B| = |D_ref|:
    X = |A n B| is hypergeometric, P(X = x) = C(a, x) C(n - a, b - x) / C(n, b),
    and J = x / (a + b - x);
  * an empty union counts as J = 1 (identical, empty drop sets), and RDA = 1
    whenever J_rand = 1 (the random baseline cannot be beaten or missed).
The adjacent-step similarity of the early-exit operator is J(t, t - 1).
"""

from fractions import Fraction
import math

import numpy as np


def drop_masks(token_pos, flags, seq_offsets):
    """Per sequence: boolean drop mask over its routable tokens (token_pos < 0)."""
    tp = np.asarray(token_pos)
    fl = np.asarray(flags)
    off = np.asarray(seq_offsets)
    out = []
    for b in range(len(off) - 1):
        lo, hi = int(off[b]), int(off[b + 1])
        routable = (fl[lo:hi] & 2) == 0
        out.append(tp[lo:hi][routable] < 0)
    return out


def jaccard(drop_t, drop_ref):
    """Eq. 10 on two boolean drop masks over the same universe."""
    inter = int(np.sum(drop_t & drop_ref))
    union = int(np.sum(drop_t | drop_ref))
    return 1.0 if union == 0 else inter / union


def _jaccard_of_counts(x, a, b):
    u = a + b - x
    return 1.0 if u == 0 else x / u


def expected_random_jaccard(n, a, b):
    """E[J] of two independent uniform subsets of sizes a, b of n items (float64).

    Sums the hypergeometric distribution term by term; each probability is
    formed in log space with math.lgamma.
    """
    if not (0 <= a <= n and 0 <= b <= n):
        raise ValueError("subset sizes outside the universe")
    lg = lambda m: math.lgamma(m + 1.0)
    log_cnb = lg(n) - lg(b) - lg(n - b)
    total = 0.0
    for x in range(max(0, a + b - n), min(a, b) + 1):
        logp = (lg(a) - lg(x) - lg(a - x)) + (lg(n - a) - lg(b - x) - lg(n - a - b + x)) - log_cnb
        total += math.exp(logp) * _jaccard_of_counts(x, a, b)
    return total


def expected_random_jaccard_exact(n, a, b):
    """The same expectation as an exact rational (small n; used to pin the float form)."""
    total = Fraction(0)
    cnb = math.comb(n, b)
    for x in range(max(0, a + b - n), min(a, b) + 1):
        u = a + b - x
        jx = Fraction(1) if u == 0 else Fraction(x, u)
        total += Fraction(math.comb(a, x) * math.comb(n - a, b - x), cnb) * jx
    return total


def rda(j, j_rand):
    """Eq. 11, with RDA = 1 when the random baseline is already 1."""
    if j_rand >= 1.0:
        return 1.0
    return (j - j_rand) / (1.0 - j_rand)


def stability(token_pos_t, token_pos_ref, flags, seq_offsets):
    """Per sequence (J, J_rand, RDA) between two timesteps' packed positions."""
    dt = drop_masks(token_pos_t, flags, seq_offsets)
    dr = drop_masks(token_pos_ref, flags, seq_offsets)
    J, JR, R = [], [], []
    for m_t, m_r in zip(dt, dr):
        n = len(m_t)
        j = jaccard(m_t, m_r)
        jr = expected_random_jaccard(n, int(m_t.sum()), int(m_r.sum()))
        J.append(j)
        JR.append(jr)
        R.append(rda(j, jr))
    return np.array(J), np.array(JR), np.array(R)
