"""Oracle: fidelity metrics between two next-base distributions -- TEST
INFRASTRUCTURE.

What is computed (Appendix "Metrics"), in float64, per position t for the
base model's distribution p_t and the FOCUS model's q_t over V categories:

  L1         sum_i |p_i - q_i|
  L2         (sum_i (p_i - q_i)^2)^(1/2)
  Hellinger  (1/sqrt 2) || sqrt(p) - sqrt(q) ||_2   (= sqrt(1 - sum_i sqrt(p_i q_i)))
  JS         KL(p || m) / 2 + KL(q || m) / 2,  m = (p + q) / 2
  KL         KL(p || q) = sum_i p_i log(p_i / q_i)       (natural log, nats)

Before any metric both distributions are clipped from below at 1e-12 and
renormalised, as the appendix prescribes for numerical stability (reading: the
clip applies to every metric and to both distributions).  Distributions may be
given as logits, turned into probabilities by the softmax definition.  The
sequence-level score is the mean of a metric over the positions of a sequence.
"""

from __future__ import annotations

import numpy as np

CLIP = 1e-12
METRICS = ("l1", "l2", "hellinger", "js", "kl")


def softmax(logits):
    """Row-wise softmax: exp(x - max) / sum."""
    x = np.asarray(logits, np.float64)
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def clip_renormalise(p):
    """Clip each probability from below at 1e-12, then divide by the row sum."""
    p = np.maximum(np.asarray(p, np.float64), CLIP)
    return p / p.sum(axis=-1, keepdims=True)


def kl(a, b):
    """KL(a || b) = sum a log(a / b), row-wise."""
    return (a * np.log(a / b)).sum(axis=-1)


def metrics(p, q):
    """The five metrics of every row of p and q ([..., V] probabilities),
    after clipping and renormalisation.  Returns [..., 5] in METRICS order."""
    p, q = clip_renormalise(p), clip_renormalise(q)
    d = p - q
    l1 = np.abs(d).sum(axis=-1)
    l2 = np.sqrt((d * d).sum(axis=-1))
    hel = np.sqrt(((np.sqrt(p) - np.sqrt(q)) ** 2).sum(axis=-1)) / np.sqrt(2.0)
    m = 0.5 * (p + q)
    js = 0.5 * kl(p, m) + 0.5 * kl(q, m)
    return np.stack([l1, l2, hel, js, kl(p, q)], axis=-1)


def metrics_from_logits(p_logits, q_logits):
    return metrics(softmax(p_logits), softmax(q_logits))


def sequence_means(per_position, cu_pos):
    """Mean of each metric over the positions [cu_pos[b], cu_pos[b+1]) of each
    sequence b (an empty sequence gives 0)."""
    cu = np.asarray(cu_pos, np.int64)
    out = np.zeros((len(cu) - 1, per_position.shape[-1]), np.float64)
    for b in range(len(cu) - 1):
        if cu[b + 1] > cu[b]:
            out[b] = per_position[cu[b]:cu[b + 1]].mean(axis=0)
    return out
