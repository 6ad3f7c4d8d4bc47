"""SnapKV prompt compaction in float64 (oracle; test infrastructure).

Appendix A.3, "SnapKV: Prompt Selection from an Observation Window" (eqs.
background-snapkv-score and background-snapkv-retention):
  * the observation window O is the prompt's last w positions;
  * every earlier position j is scored by the attention the observation
    queries pay it, u(j) = sum over i in O of alpha_{i,j}, where alpha_{i,.}
    is query i's causal attention (the keys at positions up to its own);
  * the scores are pooled over a neighbourhood of width kappa; with max
    pooling s(j) = max of u over the neighbourhood of j;
  * with budget B >= w the retained prompt is O plus the TopK_{B-w} of s over
    the earlier positions, selected separately for every head.

Readings of points the paper leaves open:
  * GQA: a KV head's u(j) sums the weights of its G query heads (as for H2O;
    parity unpinned by the paper, a convention held here).
  * The observation queries are inputs (the prefill computed them): query t
    (t = 0..w-1) sits at the t-th smallest position of the window, which is
    the w slots with the largest positions.
  * Neighbourhood of j: the candidates (slots outside O) whose positions are
    within floor(kappa/2) of pos(j), kappa odd; the window is not pooled over.
  * TopK order as for H2O: larger pooled score first, then lower position.
  * After the call the score field holds s on the candidates and 0 on the
    window; retention and compaction are H2O's with the window O (retain with
    recent = w, then the hole-fill compaction).  A unit whose prompt already
    fits the budget (L <= B) is left as it is.
"""

import numpy as np

from . import h2o
from .state import UnitState


def window_slots(pos: np.ndarray, w: int) -> np.ndarray:
    """Slots of the observation window, in increasing position order."""
    order = np.argsort(pos, kind="stable")
    return order[len(pos) - w:]


def observation_scores(Qo: np.ndarray, K: np.ndarray, pos: np.ndarray, w: int, scale: float) -> np.ndarray:
    """u over every slot (eq. background-snapkv-score, summed over the group).

    Qo: float64 [w, G, d], query t of the window's t-th position; K: [L, d].
    Returns float64 [L]; window slots receive their weights too (the caller
    uses the candidates only).
    """
    L = K.shape[0]
    obs = window_slots(pos, w)
    u = np.zeros(L, dtype=np.float64)
    for t in range(w):
        seen = pos <= pos[obs[t]]                     # causal: keys up to query t's position
        Z = scale * (K @ Qo[t].T)                     # [L, G]: every head of the group
        Z[~seen] = -np.inf
        E = np.exp(Z - Z.max(axis=0))
        u += (E / E.sum(axis=0)).sum(axis=1)
    return u


def pool_max(u: np.ndarray, pos: np.ndarray, cand: np.ndarray, kappa: int) -> np.ndarray:
    """s(j) = max of u over the candidates within kappa // 2 positions of j
    (for candidate j; 0 elsewhere)."""
    half = int(kappa) // 2
    s = np.zeros_like(u)
    idx = np.flatnonzero(cand)
    order = idx[np.argsort(pos[idx], kind="stable")]   # candidates by position
    ps = pos[order]
    lo = np.searchsorted(ps, ps - half, side="left")
    hi = np.searchsorted(ps, ps + half, side="right")
    for i, j in enumerate(order):                      # [lo, hi): |pos - pos[j]| <= half
        s[j] = u[order[lo[i]:hi[i]]].max()
    return s


def compact_prompt(st: UnitState, Qo: np.ndarray, w: int, kappa: int, budget: int, scale: float) -> dict:
    """Scores, pools, retains (eq. background-snapkv-retention) and compacts
    the unit's prompt; mutates st.  Returns u, s, keep, holes, movers, freed."""
    L = st.length
    if L <= budget:
        keep = np.ones(L, dtype=bool)
        return {"u": None, "s": None, "keep": keep, "holes": np.zeros(0, np.int64),
                "movers": np.zeros(0, np.int64), "freed": np.zeros(0, np.int64)}
    obs = window_slots(st.pos, w)
    cand = np.ones(L, dtype=bool)
    cand[obs] = False
    u = observation_scores(Qo, st.K, st.pos, w, scale)
    s = pool_max(u, st.pos, cand, kappa)
    st.u = s.copy()
    keep = h2o.retain(st.pos, st.u, budget, w)
    holes, movers, freed = h2o.compact(st, keep, budget)
    return {"u": u, "s": s, "keep": keep, "holes": holes, "movers": movers, "freed": freed}
