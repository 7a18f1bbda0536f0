"""Host-side evaluation of held-out prediction (Sec. 6): the library's
prediction pass (same_predict) counts, per test entry, how often the frozen-CPT
sampler visits the entry's true state; these helpers turn the counts into
scores and the scores into the area under the ROC curve.  Evaluation only:
no step of the sampler runs here."""
from __future__ import annotations

import numpy as np


def auc(scores, labels) -> float:
    """Area under the ROC curve of binary labels: the probability that a
    random positive scores above a random negative, ties counting one half
    (the Mann-Whitney statistic over mid-ranks)."""
    s = np.asarray(scores, dtype=np.float64).ravel()
    y = np.asarray(labels).ravel().astype(bool)
    n_pos, n_neg = int(y.sum()), int((~y).sum())
    if n_pos == 0 or n_neg == 0:
        raise ValueError("both classes are needed")
    order = np.argsort(s, kind="mergesort")
    ss = s[order]
    ranks = np.empty(len(s), dtype=np.float64)
    i = 0
    while i < len(ss):  # mid-ranks of tied runs
        j = i
        while j + 1 < len(ss) and ss[j + 1] == ss[i]:
            j += 1
        ranks[order[i:j + 1]] = 0.5 * (i + j) + 1.0
        i = j + 1
    u = ranks[y].sum() - n_pos * (n_pos + 1) / 2.0
    return float(u / (n_pos * n_neg))


def binary_scores(hits, target, n_samples, positive=1):
    """Score of 'state == positive' per test entry (target >= 0): the sampled
    frequency of the true state is an unbiased estimate of its probability
    (Sec. 6), so P(positive) is that frequency when the true state is
    positive and one minus it otherwise.  Returns (scores, labels)."""
    hits = np.asarray(hits)
    target = np.asarray(target)
    q = target >= 0
    p_true = hits[q].astype(np.float64) / float(n_samples)
    lab = target[q] == positive
    return np.where(lab, p_true, 1.0 - p_true), lab


def kl_avg(true_theta, est_theta, cpt_off, card) -> float:
    """KL_avg (Sec. 5.1): the mean over every CPT row (every distribution of
    a node given one parent configuration) of sum_x p(x) log(p(x) / q(x)),
    p the true row and q the estimated one, summing over x with q(x) > 0 (and
    p(x) log p(x) = 0 where p(x) = 0)."""
    p_all = np.asarray(true_theta, dtype=np.float64)
    q_all = np.asarray(est_theta, dtype=np.float64)
    total, rows = 0.0, 0
    for i in range(len(card)):
        K = int(card[i])
        p = p_all[cpt_off[i]:cpt_off[i + 1]].reshape(-1, K)
        q = q_all[cpt_off[i]:cpt_off[i + 1]].reshape(-1, K)
        use = (q > 0) & (p > 0)
        with np.errstate(divide="ignore", invalid="ignore"):
            terms = np.where(use, p * np.log(np.where(use, p / q, 1.0)), 0.0)
        total += terms.sum()
        rows += p.shape[0]
    return float(total / rows)
