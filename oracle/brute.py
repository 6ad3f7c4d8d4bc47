"""Independent brute-force references that pin the NumPy oracle (test infrastructure).

Everything here is pure Python over lists of floats (``math`` only, no
NumPy), so a slip in the vectorised oracle (a transposed operand, a wrong
axis, a dropped scale) cannot be repeated here by sharing code.  Only for
tiny inputs.
"""

import math


def dense_attention(q, keys, values, scale):
    """Textbook softmax attention of one query over every listed key
    (Appendix A.1, dense case S = [i]).  Returns (o, weights, lse)."""
    logits = [scale * math.fsum(qc * kc for qc, kc in zip(q, k)) for k in keys]
    top = max(logits)
    ex = [math.exp(z - top) for z in logits]
    total = math.fsum(ex)
    weights = [e / total for e in ex]
    d = len(values[0])
    o = [math.fsum(weights[j] * values[j][c] for j in range(len(values))) for c in range(d)]
    return o, weights, top + math.log(total)


def topk_indices(scores, candidates, b):
    """TopK_b over ``candidates`` by (score desc, index asc) via a full sort;
    every candidate when fewer than b."""
    ranked = sorted(candidates, key=lambda j: (-scores[j], j))
    return sorted(ranked[:b])


def h2o_retained_positions(positions, scores, budget, recent):
    """eq. background-h2o-retention by brute force over (position, score)
    pairs: the window is the min(recent, budget) largest positions, then the
    best remaining by (score desc, position asc).  Returns a sorted list of
    retained positions."""
    n = len(positions)
    if n <= budget:
        return sorted(positions)
    w = min(recent, budget)
    by_pos = sorted(range(n), key=lambda s: -positions[s])
    window = set(by_pos[:w])
    rest = [s for s in range(n) if s not in window]
    rest.sort(key=lambda s: (-scores[s], positions[s]))
    kept = list(window) + rest[:budget - w]
    return sorted(positions[s] for s in kept)


def quest_page_bound(q, page_keys, scale):
    """The page estimate of eq. background-quest-score by explicit loops."""
    d = len(q)
    total = 0.0
    for c in range(d):
        lo = min(k[c] for k in page_keys)
        hi = max(k[c] for k in page_keys)
        total += max(q[c] * lo, q[c] * hi)
    return scale * total


def pruned_slots(positions, lo, hi, keep):
    """eq. prefix-pruning by walking the slots in order: a slot stays when its
    position lies outside [lo, hi) or is one of ``keep``.  Returns the old
    slot indices that stay, in order."""
    keep = set(keep)
    return [s for s, p in enumerate(positions) if not (lo <= p < hi) or p in keep]


def interval_budget_keep(positions, scores, lo, hi, budget):
    """The ``budget`` slots of [lo, hi) with the largest scores (ties: lower
    position) by a full sort; returns their positions as a set."""
    cand = [s for s in range(len(positions)) if lo <= positions[s] < hi]
    cand.sort(key=lambda s: (-scores[s], positions[s]))
    return {positions[s] for s in cand[:budget]}
