"""Next-token sampling and its log-probability.

One draw of Alg. 1's rollout step for one sequence.  Definitions (the paper
leaves the sampler unspecified; these are the readings taken here):

* z = l / T (T = 0 means greedy and uses T = 1 for the log-probability).
* S = the top-k vocabulary ids of l ordered by (value desc, id asc); all ids
  when k = 0.
* Greedy: the lowest id among the maxima of l over S.
* Sampled: Gumbel-max, the lowest id among the maxima of z_i + g_i over S,
  g_i from the Philox counters of (seed, step, seq, i).
* logp = z_tok - ln sum_{all V} exp(z): the full-vocabulary log-softmax, no
  renormalisation to S.
"""
from __future__ import annotations

import numpy as np

from .philox import gumbel_keys


def log_softmax(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    return z - (m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True)))


def topk_set(l: np.ndarray, k: int) -> np.ndarray:
    """Ids of the k largest entries, ties broken by lower id (sorted by rank)."""
    l = np.asarray(l, np.float64)
    ids = np.arange(l.shape[0])
    order = np.lexsort((ids, -l))
    return order if k <= 0 or k >= l.shape[0] else order[:k]


def _first_argmax(v: np.ndarray) -> int:
    return int(np.flatnonzero(v == np.max(v))[0])


def sample_token(logits: np.ndarray, temperature: float, top_k: int, seed: int, step: int,
                 seq: int) -> tuple[int, float, float]:
    """Returns (token id, log-prob, decision margin).

    The margin is the gap between the winning key and the best other key in S;
    a value near zero marks a near-tie whose outcome floating-point rounding may
    legitimately decide.
    """
    l = np.asarray(logits, np.float64)
    V = l.shape[0]
    S = np.sort(topk_set(l, top_k))
    T = float(temperature)
    if T == 0.0:
        key = l[S]
        z = l
    else:
        z = l / T
        key = z[S] + gumbel_keys(seed, step, seq, V)[S]
    j = _first_argmax(key)
    tok = int(S[j])
    others = np.delete(key, j)
    margin = float(key[j] - np.max(others)) if others.size else np.inf
    logp = float(log_softmax(z)[tok])
    return tok, logp, margin
