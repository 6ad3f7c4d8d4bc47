"""Quest page selection and sparse decode in float64 (oracle; test infrastructure).

Appendix A.3, "Quest: Query-Dependent Page Selection":
  * eq. background-quest-summary: every page stores, per channel c, the
    minimum and the maximum of its keys' c-th entries;
  * eq. background-quest-score: a page's estimate for a query is 1/sqrt(d_k)
    times the sum over channels of max(q_c * min_c, q_c * max_c), an upper
    bound of every logit in the page that no single token need reach;
  * pages are ranked by the estimate and attention uses the actual KV of the
    selected pages; unselected pages stay stored; a new key updates the
    extrema of its page.
Section 3.1: selection only changes which resident entries attention reads
(eq. attention-view); nothing is evicted.

Readings of points the paper leaves open:
  * GQA: a KV head ranks pages by the *maximum* of the estimates of its G
    query heads (parity unpinned by the paper; a convention held here).
  * The page holding the newest token (the current page) is always read and
    is never a candidate; the candidates are all older pages.
  * TopK order: larger score first; equal scores -> lower page index first.
    The selected page list is returned in ascending page order.
"""

import numpy as np

from .attention import selected_attention
from .state import UnitState


def page_summaries(K: np.ndarray, length: int, page_size: int):
    """eq. background-quest-summary over slot pages of the first ``length``
    slots; a partial last page summarises the slots it holds."""
    n_pages = -(-length // page_size)
    d = K.shape[1]
    mn = np.empty((n_pages, d), dtype=np.float64)
    mx = np.empty((n_pages, d), dtype=np.float64)
    for b in range(n_pages):
        rows = K[b * page_size:min((b + 1) * page_size, length)]
        mn[b] = rows.min(axis=0)
        mx[b] = rows.max(axis=0)
    return mn, mx


def attach_summaries(st: UnitState) -> None:
    st.mn, st.mx = page_summaries(st.K, st.length, st.page_size)


def append(st: UnitState, k: np.ndarray, v: np.ndarray, p: int) -> int:
    """Adds the new token at slot L and folds its key into its page's
    extrema (a fresh page starts from the key itself)."""
    k = np.asarray(k, dtype=np.float64)
    slot = st.length
    st.K = np.vstack([st.K, k[None, :]])
    st.V = np.vstack([st.V, np.asarray(v, dtype=np.float64)[None, :]])
    st.pos = np.append(st.pos, np.int64(p))
    st.u = np.append(st.u, 0.0)
    b = slot // st.page_size
    if slot % st.page_size == 0:
        st.mn = np.vstack([st.mn, k[None, :]])
        st.mx = np.vstack([st.mx, k[None, :]])
    else:
        st.mn[b] = np.minimum(st.mn[b], k)
        st.mx[b] = np.maximum(st.mx[b], k)
    return slot


def page_bounds(q: np.ndarray, mn: np.ndarray, mx: np.ndarray, scale: float) -> np.ndarray:
    """eq. background-quest-score for every query row and page: [G, n_pages]."""
    zhat = np.empty((q.shape[0], mn.shape[0]), dtype=np.float64)
    for a in range(q.shape[0]):
        lo = q[a][None, :] * mn
        hi = q[a][None, :] * mx
        zhat[a] = np.maximum(lo, hi).sum(axis=1) * float(scale)
    return zhat


def group_page_scores(q: np.ndarray, mn: np.ndarray, mx: np.ndarray, scale: float) -> np.ndarray:
    """Per-KV-head page score: the maximum estimate over the group's heads."""
    return page_bounds(q, mn, mx, scale).max(axis=0)


def select_pages(scores: np.ndarray, n_candidates: int, top_k: int) -> np.ndarray:
    """TopK_{top_k} over pages [0, n_candidates) by (score desc, index asc);
    all candidates if there are fewer.  Returned in ascending page order."""
    cand = np.arange(int(n_candidates))
    order = np.lexsort((cand, -np.asarray(scores, dtype=np.float64)[:n_candidates]))
    return np.sort(cand[order[:int(top_k)]])


def read_set(selected: np.ndarray, length: int, page_size: int) -> np.ndarray:
    """Slots of the selected pages plus the current (newest) page."""
    cur = (length - 1) // page_size
    pages = list(int(b) for b in selected) + [cur]
    slots = [s for b in pages for s in range(b * page_size, min((b + 1) * page_size, length))]
    return np.array(slots, dtype=np.int64)


def decode_step(st: UnitState, q: np.ndarray, k: np.ndarray, v: np.ndarray,
                p: int, scale: float, top_k: int) -> dict:
    """One Quest decode step for one unit: append (summary update), rank the
    older pages with the current query, attend over the selected pages plus
    the current page.  Mutates ``st`` (append only)."""
    append(st, k, v, p)
    cur = (st.length - 1) // st.page_size
    scores = group_page_scores(q, st.mn[:cur], st.mx[:cur], scale)
    selected = select_pages(scores, cur, top_k)
    S = read_set(selected, st.length, st.page_size)
    o, lse, alpha, z = selected_attention(q, st.K, st.V, S, scale)
    return {"o": o, "lse": lse, "alpha": alpha, "z": z, "S": S,
            "scores": scores, "selected": selected, "n_candidates": cur}
