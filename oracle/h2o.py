"""H2O decode step and chunk-wise prefill eviction in float64 (oracle; test
infrastructure).

Appendix A.3, "H2O: Accumulated Scores and Online Eviction":
  * before position i is processed the available set is the previously
    retained set plus the new token, and the new token's score starts at 0;
  * attention reads the available set and every available entry's score
    grows by its attention weight (eq. background-h2o-score);
  * with budget B and a protected recent window W of at most B positions,
    the retained set is W plus the TopK_{B-|W|} of the scores over the
    remaining entries (eq. background-h2o-retention); TopK returns every
    candidate when there are fewer than requested (Table
    background-notation);
  * evicted entries leave the cache; retained scores persist.
Section 3.1 ("Method-Customized CacheManager"): physical eviction updates the
retained-slot mapping and the context length, then releases the discarded
slots.

Readings of points the paper leaves open:
  * GQA: a KV head's score grows by the *sum* of the weights of its G query
    heads (parity unpinned by the paper; a convention held here).
  * The window W is the min(w, B) slots with the largest logical positions.
  * TopK order: larger score first; equal scores -> lower logical position
    first.
  * Compacted layout (parity unpinned by the paper): slots [0, B) hold the
    retained set afterwards.  Holes are the evicted slots below B in
    ascending order, movers the retained slots at or above B in ascending
    order, and the k-th mover moves into the k-th hole with its key, value,
    position and score.  Nothing else moves.
  * Freed pages: the logical pages ceil(B/p) .. ceil(L_old/p) - 1, which hold
    no resident slot after compaction.
  * Chunked prefill (prefill_chunk): the chunk's tokens join with score 0; the
    scoring queries are the chunk's last s positions, each adding its causal
    weights (over the retained slots and the chunk up to itself) before one
    retention and compaction per chunk.
"""

import numpy as np

from .attention import selected_attention
from .state import UnitState


def append(st: UnitState, k: np.ndarray, v: np.ndarray, p: int) -> int:
    """Adds the new token at slot L with score 0; returns its slot."""
    slot = st.length
    st.K = np.vstack([st.K, np.asarray(k, dtype=np.float64)[None, :]])
    st.V = np.vstack([st.V, np.asarray(v, dtype=np.float64)[None, :]])
    st.pos = np.append(st.pos, np.int64(p))
    st.u = np.append(st.u, 0.0)
    return slot


def accumulate(u: np.ndarray, S: np.ndarray, alpha: np.ndarray) -> np.ndarray:
    """eq. background-h2o-score, summed over the G query heads of the group.

    u: float64 [L]; S: slots read; alpha: float64 [G, |S|] weights in the
    order of S.  Returns the updated copy of u.
    """
    out = np.array(u, dtype=np.float64, copy=True)
    out[np.asarray(S, dtype=np.int64)] += alpha.sum(axis=0)
    return out


def window_mask(pos: np.ndarray, budget: int, recent: int) -> np.ndarray:
    """W: the min(recent, budget) slots with the largest logical positions."""
    n = pos.shape[0]
    w = min(int(recent), int(budget), n)
    mask = np.zeros(n, dtype=bool)
    if w > 0:
        order = np.argsort(-pos, kind="stable")
        mask[order[:w]] = True
    return mask


def retain(pos: np.ndarray, u: np.ndarray, budget: int, recent: int) -> np.ndarray:
    """eq. background-h2o-retention; returns a boolean mask of retained slots.

    Scores are compared as given (float64 values; the isolation tests pass
    float32 values widened to float64 so both sides order the same numbers).
    """
    n = pos.shape[0]
    if n <= budget:
        return np.ones(n, dtype=bool)
    W = window_mask(pos, budget, recent)
    need = int(budget) - int(W.sum())
    cand = np.flatnonzero(~W)
    # Larger score first, then lower position first.
    order = np.lexsort((pos[cand], -u[cand]))
    keep = W.copy()
    keep[cand[order[:need]]] = True
    return keep


def compact(st: UnitState, keep: np.ndarray, budget: int):
    """Moves retained slots at or above B into the evicted slots below B.

    Returns (holes, movers, freed_logical_pages).  No-op when L <= B.
    """
    L = st.length
    p = st.page_size
    if L <= budget:
        return np.zeros(0, np.int64), np.zeros(0, np.int64), np.zeros(0, np.int64)
    if int(keep.sum()) != budget:
        raise ValueError("the retained set must hold exactly B slots")
    slots = np.arange(L)
    holes = slots[(slots < budget) & ~keep]
    movers = slots[(slots >= budget) & keep]
    assert holes.size == movers.size
    for h, m in zip(holes, movers):
        st.K[h] = st.K[m]
        st.V[h] = st.V[m]
        st.pos[h] = st.pos[m]
        st.u[h] = st.u[m]
    st.K = st.K[:budget].copy()
    st.V = st.V[:budget].copy()
    st.pos = st.pos[:budget].copy()
    st.u = st.u[:budget].copy()
    freed = np.arange(-(-budget // p), -(-L // p), dtype=np.int64)
    return holes, movers, freed


def decode_step(st: UnitState, q: np.ndarray, k: np.ndarray, v: np.ndarray,
                p: int, scale: float, budget: int, recent: int,
                evict: bool = True) -> dict:
    """One H2O decode step for one unit: append, attend over every resident
    slot, accumulate, then (if ``evict``) retain and compact.  Mutates ``st``.

    q: float64 [G, d] (the group's query rows); k, v: float64 [d]; p: the new
    token's logical position.
    """
    append(st, k, v, p)
    S = np.arange(st.length)
    o, lse, alpha, z = selected_attention(q, st.K, st.V, S, scale)
    st.u = accumulate(st.u, S, alpha)
    result = {"o": o, "lse": lse, "alpha": alpha, "z": z,
              "u_after_accumulate": st.u.copy(),
              "pos_after_append": st.pos.copy()}
    if evict:
        keep = retain(st.pos, st.u, budget, recent)
        holes, movers, freed = compact(st, keep, budget)
        result.update(keep=keep, holes=holes, movers=movers, freed=freed)
    return result


def prefill_chunk(st: UnitState, K: np.ndarray, V: np.ndarray, pos: np.ndarray, Qs: np.ndarray,
                  scale: float, budget: int, recent: int) -> dict:
    """H2O's chunk-wise eviction during chunked prefill for one unit (Section
    3.1: finish_step after a prefill chunk; Appendix A.3, eqs.
    background-h2o-score and background-h2o-retention; Appendix D: scores from
    a prefill scoring window).  Mutates ``st``.

    The chunk's C tokens (K, V float64 [C, d], positions ``pos`` increasing,
    all above the resident ones) join the cache with score 0.  Each scoring
    query -- the last s positions of the chunk, Qs float64 [s, G, d], query t at
    chunk position C - s + t -- reads the available set up to its own position
    (every previously retained slot and the chunk up to it) and adds its
    group's weights to those slots' scores, as the per-token recurrence does
    for one query.  Then the retained set and the compaction of a decode step.

    Readings: the scoring queries are the chunk's last s
    positions (s = C: every query of the chunk); GQA sum; window and TopK as
    for decode."""
    C = K.shape[0]
    if not 1 <= Qs.shape[0] <= C:
        raise ValueError("the scoring window must hold 1 .. C queries")
    for c in range(C):
        append(st, K[c], V[c], int(pos[c]))
    return chunk_eviction(st, C, Qs, scale, budget, recent)


def chunk_eviction(st: UnitState, C: int, Qs: np.ndarray, scale: float, budget: int, recent: int) -> dict:
    """The part of ``prefill_chunk`` after the chunk's append: the chunk is the
    unit's last C slots (score 0); its last s positions' queries Qs [s, G, d]
    add their causal weights, then the retained set and the compaction.
    Mutates ``st``."""
    s = Qs.shape[0]
    if not 1 <= s <= C <= st.length:
        raise ValueError("the scoring window must hold 1 .. C queries of a resident chunk")
    L = st.length
    for t in range(s):
        p_t = int(st.pos[L - s + t])
        S = np.flatnonzero(st.pos <= p_t)          # causal: up to the query's own position
        _, _, alpha, _ = selected_attention(Qs[t], st.K, st.V, S, scale)
        st.u = accumulate(st.u, S, alpha)
    result = {"u_after_accumulate": st.u.copy(), "pos_after_append": st.pos.copy()}
    keep = retain(st.pos, st.u, budget, recent)
    holes, movers, freed = compact(st, keep, budget)
    result.update(keep=keep, holes=holes, movers=movers, freed=freed)
    return result
