"""OmniKV cross-layer selection in float64 (oracle; test infrastructure).

Appendix A.3, "OmniKV: Selection Reuse across Layers" (eqs.
background-omnikv-selection and background-omnikv-reuse):
  * at an observation (filter) layer f, the current query of every head a
    gives each available position j its logit z^(a)_j; the position's score
    is the largest of them, s(j) = max over a of z^(a)_j;
  * the selection J is the top b positions by s over the available positions
    (those up to the current one);
  * a sparse layer assigned to f reads exactly the positions of J from its
    own cache and computes its own weights over them (selected attention,
    Appendix A.1, eq. background-selected-attention, with S = J).

Readings of points the paper leaves open:
  * heads: every query head of the request (all KV heads' groups), so J is
    one set per request, shared by its KV heads;
  * the available positions at the filter layer include the current token
    (appended before scoring), as the sparse layer's cache holds it after its
    own append;
  * TopK order: larger score first, then lower position; J is kept in
    increasing order; b >= the available positions selects all of them;
  * slots: OmniKV keeps the whole history, so every KV head of a request
    holds the same positions in the same slots, in position order; J is kept
    as slot indices.
"""

import numpy as np

from .attention import selected_attention
from .h2o import append


def position_scores(q: np.ndarray, K_heads, q_per_kv: int, scale: float) -> np.ndarray:
    """s(j) = max over the request's query heads a of scale * <q_a, k_j> with
    k_j from KV head floor(a / G) (eq. background-omnikv-selection).

    q: float64 [Hq, d]; K_heads: the request's KV heads' keys, each float64
    [L, d] with the same L.  Returns float64 [L]."""
    L = K_heads[0].shape[0]
    s = np.full(L, -np.inf)
    for a in range(q.shape[0]):
        z = scale * (K_heads[a // q_per_kv] @ q[a])
        s = np.maximum(s, z)
    return s


def select(s: np.ndarray, b: int) -> np.ndarray:
    """J = TopK_b(s): larger score first, ties to the lower position; returned
    in increasing order (every position when b >= len(s))."""
    L = s.shape[0]
    if b >= L:
        return np.arange(L, dtype=np.int64)
    order = np.lexsort((np.arange(L), -s))      # primary: -s, then the index
    return np.sort(order[:b]).astype(np.int64)


def filter_step(units, q: np.ndarray, k_new: np.ndarray, v_new: np.ndarray, p: int,
                scale: float, b: int) -> dict:
    """One decode step of an observation layer for one request: append the
    token to every KV head's cache, dense attention of each head's group, and
    the selection J from every head's logits.  Mutates the units.

    units: the request's UnitStates (one per KV head); q: float64 [Hq, d];
    k_new, v_new: float64 [Hkv, d]; p: the token's position."""
    Hkv = len(units)
    G = q.shape[0] // Hkv
    for h, st in enumerate(units):
        append(st, k_new[h], v_new[h], p)
    o = np.zeros_like(q)
    lse = np.zeros(q.shape[0])
    for h, st in enumerate(units):
        rows = slice(h * G, (h + 1) * G)
        o[rows], lse[rows], _, _ = selected_attention(q[rows], st.K, st.V, np.arange(st.length), scale)
    s = position_scores(q, [st.K for st in units], G, scale)
    return {"o": o, "lse": lse, "s": s, "J": select(s, b)}


def sparse_step(units, q: np.ndarray, k_new: np.ndarray, v_new: np.ndarray, p: int,
                scale: float, J: np.ndarray) -> dict:
    """One decode step of a sparse layer for one request: append the token,
    then each head's group attends over the slots J of its own cache (eq.
    background-omnikv-reuse).  Mutates the units."""
    Hkv = len(units)
    G = q.shape[0] // Hkv
    for h, st in enumerate(units):
        append(st, k_new[h], v_new[h], p)
    o = np.zeros_like(q)
    lse = np.zeros(q.shape[0])
    for h, st in enumerate(units):
        rows = slice(h * G, (h + 1) * G)
        o[rows], lse[rows], _, _ = selected_attention(q[rows], st.K, st.V, J, scale)
    return {"o": o, "lse": lse}
