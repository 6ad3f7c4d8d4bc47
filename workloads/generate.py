"""Seeded synthetic inputs for the decode workloads, on any torch device.

This module only draws random numbers and lays them out in the paged format
that the library's C-ABI documents:

  kv_pool     bf16  [num_pages][2][page_size][head_dim]   (K block, then V block)
  pos_pool    int32 [num_pages][page_size]                 logical position per slot
  score_pool  fp32  [num_pages][page_size]                 H2O scores (zeros)
  meta_pool   bf16  [num_pages][2][head_dim]               Quest min/max (zeros; the
                                                           cache manager fills it)
  block_table int32 [layers * units][max_pages]            unit = req * Hkv + kv_head
  lengths     int32 [layers * units]                       resident slots per unit

Slot s of a unit lives at page block_table[unit][s // page_size], row
s % page_size.  Physical pages are a seeded random permutation, so a unit's
pages are scattered over the pool.

Value recipe (the workloads' own description):
  * q, K, V ~ N(0, 1) in float32, rounded to bf16;
  * one unit vector u per (layer, KV head), shared by every request, position
    and step; every query head of the group gets q += u before rounding;
  * H2O and SnapKV workloads: a position is a heavy hitter with probability hh_rate,
    decided by a counter-based integer hash of (seed, layer, unit, position),
    so the initial context and later decode tokens follow the same rule; a
    heavy hitter's key gets += hh_shift * u before rounding to bf16 (for the
    initial context the N(0,1) draw is rounded to bf16 first);
  * Quest workload: relevant_pages random full pages per unit get
    += relevant_shift * u on all their keys;
  * ragged / retained workloads: the last `recent` positions of the context
    plus a stratified random sample (one position per stratum, so sorted and
    without repeats) of the older ones;
  * OmniKV workload: every layer keeps the whole history (slot s holds
    position s), with the heavy-hitter construction of the H2O workloads;
  * SnapKV workload: the whole prefilled prompt is resident (slot s holds
    position s) and the observation queries of its last obs_window positions
    are N(0, 1) + u, rounded to bf16, like decode queries;
  * H2O prefill workload: the chunk's `chunk` positions sit behind a
    stratified sample of the earlier ones (the retained slots, drawn like a
    retained workload with the chunk as its tail); the retained slots' scores
    are Exp(mean 0.15) (about three chunks' worth of the average weight a slot
    receives: 128 * G weight units spread over 10240 slots), the chunk's slots
    hold -1 (stale values the call replaces); the scoring queries are drawn like
    SnapKV's observation queries;
  * prefix-pruning workload: every layer keeps the whole history (slot s holds
    position s, keys N(0, 1) without heavy hitters) and the score field holds a
    scoring policy's output, U(0, 1) per slot.
No part of attention, scoring, selection or compaction is computed here.
"""

import math
from dataclasses import dataclass
from typing import Optional

import torch

from .configs import Workload

_M32 = 1 << 32


def _gen(w: Workload, tag: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(w.seed * 1_000_003 + tag * 7919 + 17)
    return g


def _mix32(x: torch.Tensor) -> torch.Tensor:
    # integer avalanche hash on values in [0, 2^32); every product < 2^59
    x = ((x ^ (x >> 16)) * 0x45D9F3B) % _M32
    x = ((x ^ (x >> 16)) * 0x45D9F3B) % _M32
    return x ^ (x >> 16)


def heavy_hitter(w: Workload, layer: int, unit: torch.Tensor, pos: torch.Tensor) -> torch.Tensor:
    """Bernoulli(hh_rate) per (layer, unit, position), as a counter-based hash."""
    if w.hh_rate <= 0:
        return torch.zeros_like(pos, dtype=torch.bool)
    key = (unit.to(torch.int64) * 0x9E3779B1 + pos.to(torch.int64) * 0x85EBCA77
           + (w.seed * 0xC2B2AE3D + layer * 0x27D4EB2F)) % _M32
    h = _mix32(_mix32(key) ^ 0x5BD1E995)
    return (h % 1_000_000) < int(round(w.hh_rate * 1_000_000))


@dataclass
class PagedInputs:
    w: Workload
    kv_pool: torch.Tensor
    pos_pool: torch.Tensor
    score_pool: Optional[torch.Tensor]
    meta_pool: Optional[torch.Tensor]
    block_table: torch.Tensor
    lengths: torch.Tensor
    max_pages: int
    ctx: torch.Tensor          # int64 [num_req]: position of the first decode token
    uvec: torch.Tensor         # float32 [layers, hkv, d]

    @property
    def units(self) -> int:
        return self.w.units_per_layer

    def layer_rows(self, layer: int) -> slice:
        return slice(layer * self.units, (layer + 1) * self.units)


@dataclass
class StepInputs:
    q: torch.Tensor        # bf16 [steps, layers, req, hq, d]
    k_new: torch.Tensor    # bf16 [steps, layers, req, hkv, d]
    v_new: torch.Tensor    # bf16 [steps, layers, req, hkv, d]
    new_pos: torch.Tensor  # int32 [steps, req]


def _contexts(w: Workload, device) -> torch.Tensor:
    if w.ctx_log_range is not None:
        lo, hi = w.ctx_log_range
        r = torch.rand(w.num_req, generator=_gen(w, 1, "cpu"), dtype=torch.float64)
        ctx = torch.floor(torch.exp(math.log(lo) + r * (math.log(hi) - math.log(lo)))).to(torch.int64)
        return ctx.clamp(lo, hi).to(device)
    return torch.full((w.num_req,), int(w.ctx), dtype=torch.int64, device=device)


def _initial_lengths(w: Workload, ctx: torch.Tensor, device) -> torch.Tensor:
    U = w.units_per_layer
    ctx_u = ctx.repeat_interleave(w.hkv)
    if w.retained_range is not None:
        lo, hi = w.retained_range
        L = torch.randint(lo, hi + 1, (U,), generator=_gen(w, 2, "cpu")).to(device)
        return torch.minimum(L, ctx_u)
    if w.initial_resident is not None:
        return torch.minimum(torch.full_like(ctx_u, int(w.initial_resident)), ctx_u)
    return ctx_u.clone()


def _positions(w: Workload, layer: int, ctx_u: torch.Tensor, L: torch.Tensor,
               cap: int, device) -> torch.Tensor:
    """int64 [U, cap] logical positions in slot order (ascending), -1 past L."""
    U = L.shape[0]
    slots = torch.arange(cap, device=device, dtype=torch.int64)[None, :].expand(U, cap)
    full = (L == ctx_u)
    recent = int(w.chunk if w.method == "h2o_prefill" else (w.recent or 0))
    n_old = (L - recent).clamp(min=0)                     # sampled older positions
    R = (ctx_u - recent).clamp(min=1)                      # older range [0, R)
    # stratum i of n_old covers [i*R//n, (i+1)*R//n); one uniform pick per stratum
    n = n_old.clamp(min=1)[:, None]
    lo = (slots * R[:, None]) // n
    hi = ((slots + 1) * R[:, None]) // n
    r = torch.rand(U, cap, generator=_gen(w, 100 + layer, device), device=device, dtype=torch.float64)
    sampled = lo + torch.floor(r * (hi - lo).to(torch.float64)).to(torch.int64)
    tail = ctx_u[:, None] - recent + (slots - n_old[:, None])
    pos = torch.where(slots < n_old[:, None], sampled, tail)
    pos = torch.where(full[:, None], slots, pos)
    return torch.where(slots < L[:, None], pos, torch.full_like(pos, -1))


def build_state(w: Workload, device, generate_values: bool = True) -> PagedInputs:
    """Initial paged cache for every layer of the workload."""
    P, d, U = w.page_size, w.head_dim, w.units_per_layer
    ctx = _contexts(w, device)
    L0 = _initial_lengths(w, ctx, device)
    if w.method == "h2o":
        cap_slots = int(max(int(L0.max()), int(w.budget)) + 1)
    elif w.method in ("snapkv", "h2o_prefill", "prune"):
        cap_slots = int(L0.max())
    elif w.method == "omnikv":
        cap_slots = int(L0.max()) + w.steps
    else:
        cap_slots = int(L0.max()) + w.steps
    max_pages = -(-cap_slots // P)
    cap = max_pages * P
    num_pages = w.layers * U * max_pages

    # each layer's pages in a region of its own (as a per-layer KV tensor),
    # scattered within it by a seeded permutation
    per_layer = U * max_pages
    gp = _gen(w, 3, device)
    perm = torch.cat([l * per_layer + torch.randperm(per_layer, generator=gp, device=device)
                      for l in range(w.layers)])
    block_table = perm.to(torch.int32).view(w.layers * U, max_pages)
    kv_pool = torch.empty((num_pages, 2, P, d), dtype=torch.bfloat16, device=device)
    pos_pool = torch.full((num_pages, P), -1, dtype=torch.int32, device=device)
    score_pool = (torch.zeros((num_pages, P), dtype=torch.float32, device=device)
                  if w.method in ("h2o", "snapkv", "h2o_prefill", "prune") else None)
    meta_pool = torch.zeros((num_pages, 2, d), dtype=torch.bfloat16, device=device) if w.method == "quest" else None
    lengths = L0.to(torch.int32).repeat(w.layers)

    g = torch.Generator(device=device)
    g.manual_seed(w.seed * 1_000_003 + 5)
    uvec = torch.randn((w.layers, w.hkv, d), generator=g, device=device, dtype=torch.float64)
    uvec = (uvec / uvec.norm(dim=-1, keepdim=True)).to(torch.float32)

    if generate_values:
        chunk = max(1, (1 << 28) // (2 * P * d))          # about 0.5 GiB of bf16 per draw
        gv = _gen(w, 4, device)
        for s in range(0, num_pages, chunk):
            kv_pool[s:s + chunk].normal_(generator=gv)

    ctx_u = ctx.repeat_interleave(w.hkv)
    kvh = torch.arange(U, device=device) % w.hkv
    for layer in range(w.layers):
        bt = block_table[layer * U:(layer + 1) * U].to(torch.int64)
        pos = _positions(w, layer, ctx_u, L0, cap, device)
        page = bt.repeat_interleave(P, dim=1)              # [U, cap]
        row = torch.arange(cap, device=device) % P
        valid = pos >= 0
        pos_pool.view(-1)[(page * P + row)[valid]] = pos[valid].to(torch.int32)
        if w.method == "h2o_prefill":
            e = torch.rand(U, cap, generator=_gen(w, 300 + layer, device), device=device, dtype=torch.float64)
            sc = (-0.15 * torch.log1p(-e)).to(torch.float32)
            old = torch.arange(cap, device=device)[None, :] < (L0 - int(w.chunk))[:, None]
            sc = torch.where(old, sc, torch.full_like(sc, -1.0))
            score_pool.view(-1)[(page * P + row)[valid]] = sc[valid]
        if w.method == "prune":
            sc = torch.rand(U, cap, generator=_gen(w, 400 + layer, device), device=device).to(torch.float32)
            score_pool.view(-1)[(page * P + row)[valid]] = sc[valid]
        if not generate_values:
            continue
        shift = None
        if w.method in ("h2o", "snapkv", "omnikv", "h2o_prefill") and w.hh_rate > 0:
            unit_ids = torch.arange(U, device=device)[:, None].expand(U, cap)
            shift = valid & heavy_hitter(w, layer, unit_ids, pos.clamp(min=0))
            amount = w.hh_shift
        elif w.method == "quest" and w.relevant_pages > 0:
            full_pages = (L0 // P)
            r = torch.rand(U, max_pages, generator=_gen(w, 200 + layer, device), device=device)
            r = torch.where(torch.arange(max_pages, device=device)[None, :] < full_pages[:, None], r,
                            torch.full_like(r, 2.0))
            chosen = r.argsort(dim=1)[:, :w.relevant_pages]
            pick = torch.zeros(U, max_pages, dtype=torch.bool, device=device)
            pick.scatter_(1, chosen, True)
            shift = pick.repeat_interleave(P, dim=1) & valid
            amount = w.relevant_shift
        if shift is not None and bool(shift.any()):
            uu, ss = shift.nonzero(as_tuple=True)
            ph = bt[uu, ss // P]
            rows = ss % P
            k = kv_pool[ph, 0, rows].to(torch.float32)
            k = k + amount * uvec[layer, kvh[uu]]
            kv_pool[ph, 0, rows] = k.to(torch.bfloat16)
    return PagedInputs(w=w, kv_pool=kv_pool, pos_pool=pos_pool, score_pool=score_pool,
                       meta_pool=meta_pool, block_table=block_table, lengths=lengths,
                       max_pages=max_pages, ctx=ctx, uvec=uvec)


def build_steps(w: Workload, state: PagedInputs, device, steps: Optional[int] = None) -> StepInputs:
    """Per-step decode inputs for every step, layer and request."""
    T = int(w.steps if steps is None else steps)
    G, d, U = w.q_per_kv, w.head_dim, w.units_per_layer
    q = torch.empty((T, w.layers, w.num_req, w.hq, d), dtype=torch.bfloat16, device=device)
    k_new = torch.empty((T, w.layers, w.num_req, w.hkv, d), dtype=torch.bfloat16, device=device)
    v_new = torch.empty_like(k_new)
    gq, gk, gv = _gen(w, 10, device), _gen(w, 11, device), _gen(w, 12, device)
    new_pos = (state.ctx[None, :] + torch.arange(T, device=device)[:, None]).to(torch.int32)
    qshift = state.uvec.repeat_interleave(G, dim=1)        # [layers, hq, d]
    unit_ids = torch.arange(U, device=device).view(w.num_req, w.hkv)
    for t in range(T):
        for layer in range(w.layers):
            x = torch.randn((w.num_req, w.hq, d), generator=gq, device=device)
            q[t, layer] = (x + qshift[layer][None]).to(torch.bfloat16)
            kx = torch.randn((w.num_req, w.hkv, d), generator=gk, device=device)
            if w.method in ("h2o", "omnikv") and w.hh_rate > 0:
                p = new_pos[t].to(torch.int64)[:, None].expand(w.num_req, w.hkv)
                hh = heavy_hitter(w, layer, unit_ids, p)
                kx = kx + w.hh_shift * hh[..., None].to(kx.dtype) * state.uvec[layer][None]
            k_new[t, layer] = kx.to(torch.bfloat16)
            v_new[t, layer] = torch.randn((w.num_req, w.hkv, d), generator=gv, device=device).to(torch.bfloat16)
    return StepInputs(q=q, k_new=k_new, v_new=v_new, new_pos=new_pos)


def build_observation(w: Workload, state: PagedInputs, device, layer: int = 0) -> torch.Tensor:
    """Observation queries of a SnapKV workload: bf16 [num_req][obs_window][hq][d],
    query t at the t-th of the prompt's last obs_window positions."""
    g = _gen(w, 20 + layer, device)
    x = torch.randn((w.num_req, w.obs_window, w.hq, w.head_dim), generator=g, device=device)
    qshift = state.uvec[layer].to(device).repeat_interleave(w.q_per_kv, dim=0)  # [hq, d]
    return (x + qshift[None, None]).to(torch.bfloat16)


def observation_queries(num_req: int, window: int, hq: int, head_dim: int, seed: int, device="cpu") -> torch.Tensor:
    """N(0, 1) observation queries, bf16 [num_req][window][hq][head_dim] (single-call tests)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed * 7919 + 23)
    return torch.randn((num_req, window, hq, head_dim), generator=g).to(torch.bfloat16).to(device)


def to_device(state: PagedInputs, device) -> PagedInputs:
    """A copy of the state with every tensor moved to ``device``."""
    def mv(t):
        return None if t is None else t.to(device)
    return PagedInputs(w=state.w, kv_pool=mv(state.kv_pool), pos_pool=mv(state.pos_pool),
                       score_pool=mv(state.score_pool), meta_pool=mv(state.meta_pool),
                       block_table=mv(state.block_table), lengths=mv(state.lengths),
                       max_pages=state.max_pages, ctx=mv(state.ctx), uvec=mv(state.uvec))


def clone_state(state: PagedInputs) -> PagedInputs:
    """A deep copy of every tensor of the state, on the same device."""
    def cp(t):
        return None if t is None else t.clone()
    return PagedInputs(w=state.w, kv_pool=cp(state.kv_pool), pos_pool=cp(state.pos_pool),
                       score_pool=cp(state.score_pool), meta_pool=cp(state.meta_pool),
                       block_table=cp(state.block_table), lengths=cp(state.lengths),
                       max_pages=state.max_pages, ctx=cp(state.ctx), uvec=cp(state.uvec))


def unit_slots(state: PagedInputs, unit_row: int, length: Optional[int] = None):
    """Reads one unit's slots [0, L) back in slot order, as CPU tensors:
    (K bf16 [L, d], V bf16 [L, d], pos int32 [L], u fp32 [L] or None)."""
    P = state.w.page_size
    L = int(state.lengths[unit_row]) if length is None else int(length)
    bt = state.block_table[unit_row].to(torch.int64)
    s = torch.arange(L, device=bt.device)
    page, row = bt[s // P], s % P
    K = state.kv_pool[page, 0, row].cpu()
    V = state.kv_pool[page, 1, row].cpu()
    pos = state.pos_pool[page, row].cpu()
    u = None if state.score_pool is None else state.score_pool[page, row].cpu()
    return K, V, pos, u


def isolated_units(lengths, max_pages: int, head_dim: int, seed: int, *, num_kv_heads: int = 1,
                   position_mode: str = "contiguous", score_levels: int = 0,
                   with_scores: bool = True, with_meta: bool = False, device="cpu") -> PagedInputs:
    """Units with given resident lengths for single-call tests.

    position_mode: "contiguous" (slot s has position s + offset), "shuffled"
    (distinct random positions in random slot order, as compaction leaves them),
    "gapped" (sorted random distinct positions, so recent positions are not
    contiguous) or "permuted" (positions 0 .. L-1 in random slot order: a
    contiguous recent run scattered over the slots, as steady-state eviction
    leaves it).  score_levels > 0 draws scores from that many distinct values
    (many exact ties); 0 draws continuous uniform scores.  Scores are float32.
    """
    U = len(lengths)
    P = 16
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    num_pages = U * max_pages + 7                          # a few pages nobody owns
    perm = torch.randperm(num_pages, generator=g)[:U * max_pages]
    block_table = perm.to(torch.int32).view(U, max_pages)
    kv_pool = torch.randn((num_pages, 2, P, head_dim), generator=g).to(torch.bfloat16)
    pos_pool = torch.full((num_pages, P), -1, dtype=torch.int32)
    score_pool = torch.zeros((num_pages, P), dtype=torch.float32) if with_scores else None
    for u, L in enumerate(lengths):
        L = int(L)
        if position_mode == "contiguous":
            pos = torch.arange(L, dtype=torch.int64) + 1000 * u
        elif position_mode == "shuffled":
            pos = torch.randperm(4 * L + 8, generator=g)[:L]
        elif position_mode == "gapped":
            pos = torch.sort(torch.randperm(4 * L + 8, generator=g)[:L]).values
        elif position_mode == "permuted":
            pos = torch.randperm(L, generator=g).to(torch.int64)
        else:
            raise ValueError(position_mode)
        s = torch.arange(L)
        ph = block_table[u, s // P].to(torch.int64)
        pos_pool[ph, s % P] = pos.to(torch.int32)
        if with_scores:
            if score_levels > 0:
                sc = torch.randint(0, score_levels, (L,), generator=g).to(torch.float32) / score_levels
            else:
                sc = torch.rand(L, generator=g, dtype=torch.float32)
            score_pool[ph, s % P] = sc
    meta_pool = torch.zeros((num_pages, 2, head_dim), dtype=torch.bfloat16) if with_meta else None
    w = Workload(-1, "isolated", "h2o", num_req=U // num_kv_heads, hq=num_kv_heads, hkv=num_kv_heads,
                 head_dim=head_dim, layers=1, steps=0, ctx=0, seed=seed)
    st = PagedInputs(w=w, kv_pool=kv_pool, pos_pool=pos_pool, score_pool=score_pool,
                     meta_pool=meta_pool, block_table=block_table,
                     lengths=torch.tensor([int(L) for L in lengths], dtype=torch.int32),
                     max_pages=max_pages, ctx=torch.zeros(U // num_kv_heads, dtype=torch.int64),
                     uvec=torch.zeros(1, num_kv_heads, head_dim))
    return to_device(st, device)
