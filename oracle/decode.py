"""Decode-phase cache updates (H2O, TOVA), one (sequence, layer, KV head) at a time (float64).

Test infrastructure only (see the package docstring).

This is the incremental-update handler of the common operator interface
(Section 3.4) for H2O, whose retention rule keeps heavy hitters of accumulated
attention (Section 2.1).  The cache keeps a fixed capacity C: every step one
token arrives and one leaves.

Readings taken where the paper is silent:
  * the cache starts from the prefill H2O selection, each slot's accumulated
    score seeded with its unpooled group-mean window score;
  * step with new position p: the new key/value joins the C cached entries;
    each of the G query heads of the group attends over those C+1 entries
    (softmax of q.k / sqrt(d)); every entry's accumulated score grows by the
    group mean of its probabilities (the new entry starts from 0);
  * the r most recent positions p-r+1..p are protected (r = floor(C * num/den));
    among the other entries the smallest accumulated score is evicted, ties to
    the smallest position; the new token takes the victim's slot (if the new
    token itself is the victim, the slots keep their old tokens).

TOVA (Section 2.1 names it: eviction by the attention of the current query; the
paper's matched study runs it in decode only, which is the reading here):
  * step with new position p: the G query heads of the group attend over the C
    cached entries plus the new one; an entry's score is the group mean of its
    probabilities at this step alone (nothing accumulates across steps);
  * every one of the C+1 entries is a candidate (no recency protection); the
    smallest score is evicted, ties to the smallest position; the new token
    takes the victim's slot (if it is the victim itself, nothing changes).
"""
from __future__ import annotations

import numpy as np


def h2o_step(k_cache, pos, acc, q_t, k_t, p: int, recent: int):
    """One step for one KV head.

    k_cache [C, d] float64, pos [C] int, acc [C] float64, q_t [G, d] float64, k_t [d] float64.
    Returns (acc_all [C+1] accumulated scores before eviction, victim entry index in
    [0, C] where C denotes the new token, candidates mask [C+1]).
    """
    C, d = k_cache.shape
    keys = np.concatenate([k_cache, k_t[None, :]], axis=0)           # [C+1, d]
    logits = (q_t @ keys.T) / np.sqrt(d)                             # [G, C+1]
    m = logits.max(axis=1, keepdims=True)
    probs = np.exp(logits - m)
    probs /= probs.sum(axis=1, keepdims=True)
    acc_all = np.concatenate([acc, [0.0]]) + probs.mean(axis=0)
    pos_all = np.concatenate([np.asarray(pos, dtype=np.int64), [p]])
    cand = pos_all <= p - recent
    if not cand.any():
        raise ValueError("no evictable entry")
    # argmin acc among candidates, ties -> smallest position
    order = sorted(np.flatnonzero(cand), key=lambda e: (acc_all[e], pos_all[e]))
    return acc_all, int(order[0]), cand


def apply_step(k_cache, v_cache, pos, acc, acc_all, victim: int, k_t, v_t, p: int):
    """Write the new token into the victim's slot (in place); returns nothing."""
    C = k_cache.shape[0]
    acc[:] = acc_all[:C]
    if victim < C:
        k_cache[victim] = k_t
        v_cache[victim] = v_t
        pos[victim] = p
        acc[victim] = acc_all[C]


def tova_step(k_cache, pos, q_t, k_t, p: int):
    """One TOVA step for one KV head.

    k_cache [C, d] float64, pos [C] int, q_t [G, d] float64, k_t [d] float64.
    Returns (score [C+1] group-mean probabilities of this step, victim entry index in [0, C]
    where C denotes the new token).
    """
    C, d = k_cache.shape
    keys = np.concatenate([k_cache, k_t[None, :]], axis=0)           # [C+1, d]
    logits = (q_t @ keys.T) / np.sqrt(d)                             # [G, C+1]
    m = logits.max(axis=1, keepdims=True)
    probs = np.exp(logits - m)
    probs /= probs.sum(axis=1, keepdims=True)
    score = probs.mean(axis=0)
    pos_all = np.concatenate([np.asarray(pos, dtype=np.int64), [p]])
    # argmin score over all C+1 entries, ties -> smallest position
    victim = min(range(C + 1), key=lambda e: (score[e], pos_all[e]))
    return score, int(victim)


def apply_tova(k_cache, v_cache, pos, victim: int, k_t, v_t, p: int):
    """Write the new token into the victim's slot (in place); returns nothing."""
    if victim < k_cache.shape[0]:
        k_cache[victim] = k_t
        v_cache[victim] = v_t
        pos[victim] = p
