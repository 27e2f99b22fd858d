"""Prefill prompt-cache compression, one layer at a time (float64).

Test infrastructure only (see the package docstring).

The plan of Eq. 1 (Section 3.1) gives each layer an operator and a nominal
capacity b; this module is the operator side for the prefill phase, i.e. the
prompt-compression handler of the common operator interface (Section 3.4).
The retention rules are the ones the paper composes (Section 2.1 names their
families): SnapKV ranks prompt positions by the attention the last few prompt
queries give them, H2O ranks by attention summed over queries, TOVA ranks by
the attention of the newest query alone, StreamingLLM keeps the first few
positions plus the newest ones, and Full evicts nothing.  Section 3.3 fixes
that SnapKV's capacity includes its observation window.

Notation per (sequence, layer): Hq query heads, Hkv KV heads, G = Hq / Hkv,
head_dim d, context L, window w.  Arrays are float64 holding exact bf16 values.

Readings taken where the paper is silent:
  * causal mask inside the window: window row i sits at position L-w+i and
    sees keys 0..L-w+i; the softmax runs over every visible key;
  * logit scale 1/sqrt(d);
  * GQA mapping: query head hq reads KV head hq // G;
  * SnapKV: window sum, max-pool (stride 1, clipped to the prefix [0, L-w)),
    then mean over the query group; top-(b-w) over the prefix plus the window;
    b <= w keeps the last b positions;
  * H2O prefill: the same window sum with no pooling, group mean; r = floor(b *
    num / den) most recent positions kept (num/den = 1/2 by default) and the
    top-(b-r) of [0, L-r);
  * H2O with full-span accumulation (H2O_FULL): the same with every prompt
    position as a query (the window is the whole prompt, so q holds L rows):
    S[j] is the group mean of the attention key j receives from all queries
    t >= j, H2O's accumulated attention over the prompt; same selection as H2O;
  * TOVA (prefill): the prompt's last query (position L-1, the last row of
    the window block) alone: S[j] is the group mean of its softmax over every
    key 0..L-1; the top-b of [0, L) are kept, nothing is forced (Appendix C
    runs the standalone TOVA baseline in both phases);
  * StreamingLLM: s0 = min(n_sink, b) first positions and the b-s0 last;
  * any rule with b >= L keeps all L positions;
  * top-k order: value descending, then position ascending, on the float64
    scores;
  * retained positions are returned in ascending order.
"""
from __future__ import annotations

import numpy as np

FULL, STREAMING, SNAPKV, H2O = 0, 1, 2, 3
TOVA = 4   # decode: oracle.decode.tova_step; prefill: the last query's attention
H2O_FULL = 5
RULE_NAMES = {FULL: "full", STREAMING: "streaming", SNAPKV: "snapkv", H2O: "h2o", TOVA: "tova",
              H2O_FULL: "h2o_full"}


def bf16_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- window attention

def window_logits(q: np.ndarray, k: np.ndarray) -> np.ndarray:
    """z[hq, i, j] = q[hq, i] . k[hq // G, j] / sqrt(d); keys after row i's position are -inf.

    q: [Hq, w, d] (the last w prompt positions' queries), k: [Hkv, L, d].
    """
    Hq, w, d = q.shape
    Hkv, L, _ = k.shape
    G = Hq // Hkv
    z = np.empty((Hq, w, L))
    for hq in range(Hq):
        z[hq] = (q[hq] @ k[hq // G].T) / np.sqrt(d)
    row_pos = L - w + np.arange(w)
    hidden = np.arange(L)[None, :] > row_pos[:, None]
    z[:, hidden] = -np.inf
    return z


def softmax_rows(z: np.ndarray) -> np.ndarray:
    """Row softmax over the last axis; -inf entries get probability 0."""
    m = z.max(axis=-1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=-1, keepdims=True)


def window_scores(q: np.ndarray, k: np.ndarray) -> np.ndarray:
    """A[hq, j] = sum over the w window rows of the attention probability of key j. [Hq, L]"""
    return softmax_rows(window_logits(q, k)).sum(axis=1)


def max_pool_prefix(a: np.ndarray, kernel: int, n: int) -> np.ndarray:
    """Stride-1 max-pool over positions [0, n) of the last axis, window clipped at 0 and n.

    out[..., j] = max(a[..., t] for t in [j - kernel//2, j + kernel//2] and 0 <= t < n).
    """
    half = kernel // 2
    x = a[..., :n]
    padded = np.full(x.shape[:-1] + (n + 2 * half,), -np.inf)
    padded[..., half:half + n] = x
    out = np.full(x.shape, -np.inf)
    for off in range(2 * half + 1):
        out = np.maximum(out, padded[..., off:off + n])
    return out


def group_mean(a: np.ndarray, G: int) -> np.ndarray:
    """Mean over the G query heads of each KV head: [Hq, n] -> [Hq // G, n]."""
    Hq = a.shape[0]
    return a.reshape(Hq // G, G, *a.shape[1:]).mean(axis=1)


# ---------------------------------------------------------------- selection

def topk_positions(scores: np.ndarray, k: int) -> np.ndarray:
    """The first k positions in (value descending, position ascending) order, sorted ascending."""
    s = np.asarray(scores, dtype=np.float64)
    order = np.argsort(-s, kind="stable")
    return np.sort(order[:k]).astype(np.int64)


def h2o_recent(b: int, num: int, den: int) -> int:
    """Recent-token share of an H2O capacity b: floor(b * num / den)."""
    return (b * num) // den


def rule_layout(rule: int, b: int, L: int, w: int, n_sink: int = 4, num: int = 1, den: int = 2):
    """(cand_end, k, forced_lo, forced_hi) for one layer, or None when every position is kept.

    Retained set = TopK_k(S[0:cand_end]) + [forced_lo, forced_hi); for StreamingLLM the
    'top-k' part is the closed-form sink prefix [0, k) (cand_end == k).
    """
    if rule == FULL or b >= L:
        return None
    if rule == STREAMING:
        s0 = min(n_sink, b)
        return (s0, s0, L - (b - s0), L)
    if rule == SNAPKV:
        if b <= w:
            return (0, 0, L - b, L)
        return (L - w, b - w, L - w, L)
    if rule in (H2O, H2O_FULL):
        r = h2o_recent(b, num, den)
        return (L - r, b - r, L - r, L)
    if rule == TOVA:
        return (L, b, L, L)
    raise ValueError("unknown rule")


def evict_layer(rule: int, b: int, q_bits, k_bits, v_bits, *, window: int, pool_kernel: int = 7,
                n_sink: int = 4, recent_num: int = 1, recent_den: int = 2):
    """Prompt compression of one (sequence, layer).

    q_bits [Hq, w, d] ([Hq, L, d] for H2O_FULL: every position's query; TOVA reads its last
    row, the query of position L-1), k_bits / v_bits [Hkv, L, d] as bf16 bit patterns (uint16).
    Returns dict:
      idx    [Hkv, b_eff] int64, ascending retained positions
      k_out, v_out [Hkv, b_eff, d] uint16 (bit copies of the retained rows)
      scores [Hkv, cand_end] float64 candidate scores (None for unscored rules)
      layout (cand_end, k, forced_lo, forced_hi) or None
      acc    [Hkv, b_eff] float64: unpooled group-mean score at each retained position
             (the window score for SnapKV / H2O, H2O's accumulated attention; the full-span
             score for H2O_FULL; the last query's attention for TOVA; zeros for unscored rules)
    """
    k_bits = np.asarray(k_bits)
    Hkv, L, d = k_bits.shape
    w = window
    if not (1 <= w <= L):
        raise ValueError("window must be in [1, L]")
    b_eff = L if rule == FULL else min(b, L)
    layout = rule_layout(rule, b, L, w, n_sink, recent_num, recent_den)
    scored = rule in (SNAPKV, H2O, H2O_FULL, TOVA)
    if rule == H2O_FULL and np.asarray(q_bits).shape[1] != L:
        raise ValueError("H2O_FULL takes the queries of all L positions")

    A = None
    if scored:
        q = bf16_to_f64(q_bits)
        if rule == TOVA:
            q = q[:, -1:, :]                        # the query of position L-1 only
        k = bf16_to_f64(k_bits)
        G = q.shape[0] // Hkv
        A = window_scores(q, k)                     # [Hq, L]
        S_unpooled = group_mean(A, G)               # [Hkv, L]

    scores = None
    if layout is None:
        idx = np.tile(np.arange(L, dtype=np.int64), (Hkv, 1))
        if scored:
            if rule == SNAPKV:
                scores = group_mean(max_pool_prefix(A, pool_kernel, L - w), G)
            else:
                scores = S_unpooled
    else:
        cand_end, kk, lo, hi = layout
        forced = np.arange(lo, hi, dtype=np.int64)
        rows = []
        if rule == STREAMING:
            for h in range(Hkv):
                rows.append(np.concatenate([np.arange(kk, dtype=np.int64), forced]))
        else:
            if rule == SNAPKV:
                scores = group_mean(max_pool_prefix(A, pool_kernel, cand_end), G)
            else:
                scores = S_unpooled[:, :cand_end]
            for h in range(Hkv):
                sel = topk_positions(scores[h], kk)
                rows.append(np.concatenate([sel, forced]))
        idx = np.stack(rows)
    assert idx.shape == (Hkv, b_eff)

    v_bits = np.asarray(v_bits)
    k_out = np.stack([k_bits[h, idx[h]] for h in range(Hkv)])
    v_out = np.stack([v_bits[h, idx[h]] for h in range(Hkv)])
    if scored:
        acc = np.stack([S_unpooled[h, idx[h]] for h in range(Hkv)])
    else:
        acc = np.zeros((Hkv, b_eff))
    return {"idx": idx, "k_out": k_out, "v_out": v_out, "scores": scores, "layout": layout,
            "acc": acc}


def evict_route(rules, budgets, layer_inputs, *, window: int, pool_kernel: int = 7, n_sink: int = 4,
                recent_num: int = 1, recent_den: int = 2):
    """Apply a prefill route (one rule and capacity per layer, Eq. 1) to a list of per-layer inputs.

    layer_inputs[l] is a dict with "q", "k", "v" bit arrays for one sequence.
    """
    return [evict_layer(r, b, x["q"], x["k"], x["v"], window=window, pool_kernel=pool_kernel,
                        n_sink=n_sink, recent_num=recent_num, recent_den=recent_den)
            for r, b, x in zip(rules, budgets, layer_inputs)]
