"""Interval prefix-cache pruning in float64 (oracle; test infrastructure).

Section 3.2, "Sparsity-Based Prefix-Cache Pruning" (eq. prefix-pruning), and
Appendix C.2, "Pruning Metadata and Cache Operations":
  * the application names a history interval [lo, hi) of zero-based logical
    positions, T = {i | lo <= i < hi};
  * a scoring policy picks the positions I to keep inside it, a subset of the
    resident positions in T, and hands them over as a mask; the appendix also
    lets the caller give a retained-token budget (zero removes every entry of
    the interval);
  * the logical prefix is unchanged and the resident set becomes
    R' = (R minus T) union I; the slots outside R' are released.

Readings of points the paper leaves open:
  * the mask is indexed by position offset inside the interval (entry i says
    whether position lo + i is kept); entries for positions that are not
    resident have nothing to keep and are ignored;
  * budget selection: the `budget` resident slots of T with the largest scores
    (the unit's score field: accumulated H2O scores or a policy's scores),
    equal scores keeping the lower position; every slot of T when it holds
    fewer, none for a budget of 0;
  * slot layout afterwards (parity unpinned by the paper, which records
    retained offsets inside each logical block): the retained slots keep their
    relative slot order and occupy slots 0 .. |R'| - 1, each with its key,
    value, logical position (not renumbered, so P' = P) and score;
  * released pages: the logical pages ceil(|R'| / p) .. ceil(L / p) - 1, which
    hold no resident slot afterwards;
  * the interval need not be page-aligned (the slots are dense per unit here);
  * Quest page summaries, when the unit keeps them, are rebuilt from the
    pruned slots (eq. background-quest-summary over the new pages).
"""

import numpy as np

from .quest import attach_summaries
from .state import UnitState


def in_interval(pos: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """Membership of each slot's logical position in T = [lo, hi)."""
    pos = np.asarray(pos, dtype=np.int64)
    return (pos >= int(lo)) & (pos < int(hi))


def mask_selection(st: UnitState, lo: int, hi: int, mask: np.ndarray) -> np.ndarray:
    """I from a policy's mask over the interval: the resident positions p in T
    with mask[p - lo] nonzero.  Returns the kept positions, increasing."""
    mask = np.asarray(mask)
    if mask.shape[0] < max(int(hi) - int(lo), 0):
        raise ValueError("the mask must cover the interval")
    inside = st.pos[in_interval(st.pos, lo, hi)]
    keep = [int(p) for p in inside if mask[int(p) - int(lo)] != 0]
    return np.array(sorted(keep), dtype=np.int64)


def budget_selection(st: UnitState, lo: int, hi: int, budget: int) -> np.ndarray:
    """I = the `budget` resident positions of T with the largest scores (ties:
    lower position first); all of them if fewer, none for budget 0.  Returns
    the kept positions, increasing."""
    if budget < 0:
        raise ValueError("the budget must be >= 0")
    sel = np.flatnonzero(in_interval(st.pos, lo, hi))
    order = np.lexsort((st.pos[sel], -st.u[sel]))     # larger score, then lower position
    kept = st.pos[sel[order[:int(budget)]]]
    return np.sort(kept).astype(np.int64)


def retained_positions(R, lo: int, hi: int, I) -> set:
    """eq. prefix-pruning as sets: R' = (R minus T) union I, with I a subset of
    R intersected with T."""
    R = {int(p) for p in R}
    T = {p for p in R if lo <= p < hi}
    I = {int(p) for p in I}
    if not I <= T:
        raise ValueError("I must hold resident positions of the interval")
    return (R - T) | I


def prune(st: UnitState, lo: int, hi: int, I) -> dict:
    """Applies the pruning to one unit: the slots whose positions leave R' are
    removed and the retained ones close up in their slot order.  Mutates
    ``st``; returns the kept mask over the old slots, the destination slot of
    each kept one and the released logical pages."""
    Rp = retained_positions(st.pos.tolist(), lo, hi, I)
    L = st.length
    keep = np.array([int(p) in Rp for p in st.pos], dtype=bool)
    dest = np.cumsum(keep) - 1                         # rank among the kept slots
    st.K = st.K[keep].copy()
    st.V = st.V[keep].copy()
    st.pos = st.pos[keep].copy()
    st.u = st.u[keep].copy()
    if st.mn is not None:
        attach_summaries(st)
    p = st.page_size
    freed = np.arange(-(-st.length // p), -(-L // p), dtype=np.int64)
    return {"keep": keep, "dest": dest[keep], "freed": freed}
