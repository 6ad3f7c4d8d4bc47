"""Selected-set decode attention in float64 (oracle; test infrastructure).

Follows Appendix A.1, eq. background-selected-attention: for a query q and a
non-empty read set S, the logit of key j is the dot product of q and k_j
scaled by 1/sqrt(d_k), the weights are the softmax of those logits over S
only, and the output is the weighted sum of the values in S.

GQA (Appendix A.1, "MHA, MQA, and GQA"): query head a reads KV head g(a).
This repository takes g(a) = floor(a / G) with G = Hq / Hkv, so the G query
heads of one KV head are contiguous.  One call here handles one KV head's
unit: the G query heads of its group against that head's keys and values.

The softmax scale is passed in by the caller (the same float32 value the GPU
path uses) instead of being recomputed here, so both sides scale by the same
number.
"""

import numpy as np


def group_heads(kv_head: int, q_per_kv: int) -> np.ndarray:
    """Query heads a with g(a) = kv_head under g(a) = floor(a / G)."""
    return np.arange(kv_head * q_per_kv, (kv_head + 1) * q_per_kv)


def selected_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray,
                       S: np.ndarray, scale: float):
    """Attention of G query rows over the key/value rows listed in ``S``.

    q: float64 [G, d]; K, V: float64 [L, d] (one row per resident slot);
    S: int array of slot indices (non-empty, no repeats); scale: the logit
    scale (1/sqrt(d_k) rounded to float32 by the caller).

    Returns (o, lse, alpha, z):
      o     float64 [G, d]   output per query head
      lse   float64 [G]      natural log of sum_j exp(z_j) over S
      alpha float64 [G, |S|] normalised weights, in the order of S
      z     float64 [G, |S|] logits, in the order of S
    """
    S = np.asarray(S, dtype=np.int64)
    if S.size == 0:
        raise ValueError("the read set must be non-empty")
    if np.unique(S).size != S.size:
        raise ValueError("the read set lists a slot twice")
    Ks = K[S]
    Vs = V[S]
    z = (q @ Ks.T) * float(scale)
    m = z.max(axis=1, keepdims=True)
    w = np.exp(z - m)
    l = w.sum(axis=1, keepdims=True)
    alpha = w / l
    o = alpha @ Vs
    lse = (m + np.log(l))[:, 0]
    return o, lse, alpha, z
