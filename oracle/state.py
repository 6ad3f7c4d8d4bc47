"""Logical per-unit cache state used by the oracle (test infrastructure).

A unit is one (layer, request, KV head).  The oracle keeps a unit's cache as
plain arrays in *slot order*: slot s holds one resident token's key, value,
logical position and (for H2O) accumulated score.  There are no pages and no
block tables here; the paged layout (Appendix A.2, "Logical Positions and
Physical Blocks": block floor((j-1)/p), offset (j-1) mod p for 1-based j, or
slot // p and slot % p with 0-based slots) is the GPU path's business, and
the tests gather the GPU's pages back into slot order before comparing.

Section 3.1 ("Method-Customized CacheManager") and Appendix A.2 note that
after compaction physical offsets no longer follow logical positions, which
is why every slot carries its logical position ``pos``.
"""

from dataclasses import dataclass, field
from typing import Optional

import numpy as np


@dataclass
class UnitState:
    K: np.ndarray                 # float64 [L, d]
    V: np.ndarray                 # float64 [L, d]
    pos: np.ndarray               # int64 [L], logical position of each slot
    u: np.ndarray                 # float64 [L], H2O accumulated score
    page_size: int = 16
    # Quest page summaries over slot pages (slot // page_size); None if unused.
    mn: Optional[np.ndarray] = field(default=None)   # float64 [n_pages, d]
    mx: Optional[np.ndarray] = field(default=None)   # float64 [n_pages, d]

    @property
    def length(self) -> int:
        return int(self.pos.shape[0])

    @property
    def head_dim(self) -> int:
        return int(self.K.shape[1])

    def copy(self) -> "UnitState":
        return UnitState(
            K=self.K.copy(), V=self.V.copy(), pos=self.pos.copy(),
            u=self.u.copy(), page_size=self.page_size,
            mn=None if self.mn is None else self.mn.copy(),
            mx=None if self.mx is None else self.mx.copy())


def new_unit(K, V, pos, u=None, page_size: int = 16) -> UnitState:
    """Wraps float64 arrays (copies them) into a UnitState; u defaults to 0."""
    K = np.array(K, dtype=np.float64)
    V = np.array(V, dtype=np.float64)
    pos = np.array(pos, dtype=np.int64)
    if u is None:
        u = np.zeros(pos.shape[0], dtype=np.float64)
    u = np.array(u, dtype=np.float64)
    if K.shape != V.shape or K.shape[0] != pos.shape[0] or u.shape != pos.shape:
        raise ValueError("K, V, pos and u must agree on the number of slots")
    return UnitState(K=K, V=V, pos=pos, u=u, page_size=page_size)
