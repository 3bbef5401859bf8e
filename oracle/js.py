"""CPU oracle of the Jensen--Shannon functional distance.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg use this module; the product path never imports it.

What it computes (Sec. 4.4, JS distance; Appendix D.2, JS functional
disagreement), in float64 and in the log domain, for workers m = 0..M-1 and
tokens u of a fixed batch, from logits z (the model outputs at u):

    log p_m(u)   = z_m(u) - logsumexp(z_m(u))      full-vocabulary log-softmax
    log pbar(u)  = zbar(u) - logsumexp(zbar(u))    the parameter-averaged model
    T(u)         = the k tokens of largest pbar(u) (the paper uses k = 100,
                   recomputed for every u); equal logits: lower token index first
    log mix_i    = log((p_m,i + pbar_i) / 2)
    JS_m(u)      = 1/2 sum_{i in T(u)} p_m,i (log p_m,i - log mix_i)
                 + 1/2 sum_{i in T(u)} pbar_i (log pbar_i - log mix_i)
    d_m(u)       = sqrt(JS_m(u) / log 2)           normalized JS distance
    CD_JS        = mean over m and u of d_m(u)

Reading taken: the probabilities are those of the full softmax and only the
sum is restricted to T(u) (no renormalisation over T).  Every term of the sum
is non-negative, so the restricted sum is a lower bound of the full one and
equals it at k = vocabulary size.
"""

from __future__ import annotations

import numpy as np
from scipy.special import logsumexp

LOG2 = np.log(2.0)


def top_k_indices(zbar, k):
    """Indices of the k largest logits, ties broken by lower index; returned
    in ascending index order."""
    zbar = np.asarray(zbar, np.float64)
    order = np.lexsort((np.arange(zbar.size), -zbar))  # by value descending, then index ascending
    return np.sort(order[:k])


def js_distance_token(z_worker, z_avg, k):
    """d_m(u) for one worker and one token (float64)."""
    zw = np.asarray(z_worker, np.float64)
    za = np.asarray(z_avg, np.float64)
    lp = zw - logsumexp(zw)
    la = za - logsumexp(za)
    t = top_k_indices(za, k)
    lp, la = lp[t], la[t]
    with np.errstate(invalid="ignore"):
        lmix = np.logaddexp(lp, la) - LOG2
        # A token of probability 0 on one side contributes 0 to that side's
        # KL term (0 log 0 = 0); masked tokens have logit -inf.
        tp = np.where(np.isneginf(lp), 0.0, np.exp(lp) * (lp - lmix))
        ta = np.where(np.isneginf(la), 0.0, np.exp(la) * (la - lmix))
    js = 0.5 * np.sum(tp) + 0.5 * np.sum(ta)
    return float(np.sqrt(max(js, 0.0) / LOG2))


def js_distances(z_workers, z_avg, k=100):
    """z_workers [M][U][K], z_avg [U][K] (any float dtype, or bf16 bits as
    uint16 -- pass decoded values).  Returns (d [M][U], mean over tokens [M],
    top-k index sets [U][k])."""
    zw = np.asarray(z_workers)
    za = np.asarray(z_avg)
    M, U, K = zw.shape
    d = np.zeros((M, U), np.float64)
    tops = np.zeros((U, min(k, K)), np.int64)
    for u in range(U):
        tops[u] = top_k_indices(za[u], k)
        for m in range(M):
            d[m, u] = js_distance_token(zw[m, u], za[u], k)
    return d, d.mean(axis=1), tops
