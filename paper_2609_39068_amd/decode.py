"""Decode-step drivers: the order in which one layer's step calls the C-ABI.

The paper's lifecycle (Section 3.1, "Fine-Grained Lifecycle Hooks") runs
Quest's query-dependent page selection in build_decode_selection, before
attention, and H2O's score update plus online eviction in finish_step, after
it; OmniKV selects at its observation layers and the later layers reuse that
selection.  These drivers issue exactly that sequence of library calls on the
current stream, with workspaces allocated once up front; they never wait for
the device.
"""

import torch

from . import _binding as se


class H2ODecoder:
    """One layer's H2O decode step: append + attention + fused score update
    (se_decode_attend), then retention and compaction (se_evict_compact)."""

    def __init__(self, view: se.KVView, q_per_kv: int, scale: float, budget: int, recent: int,
                 max_len: int, device, report_freed: bool = False, ws=None, dev_err=None):
        """``ws`` / ``dev_err`` may be shared by decoders whose calls run one
        after another on one stream (e.g. the layers of a model)."""
        self.view, self.G, self.scale = view, q_per_kv, scale
        self.budget, self.recent, self.max_len = budget, recent, max_len
        self.ws = ws if ws is not None else self.workspace(view, q_per_kv, max_len, device)
        self.dev_err = dev_err if dev_err is not None else torch.zeros(1, dtype=torch.int32, device=device)
        self.freed = None
        self.freed_count = None
        if report_freed:
            self.freed = torch.zeros((view.num_units, view.struct.max_pages), dtype=torch.int32,
                                     device=device)
            self.freed_count = torch.zeros(view.num_units, dtype=torch.int32, device=device)

    @staticmethod
    def workspace(view: se.KVView, q_per_kv: int, max_len: int, device) -> torch.Tensor:
        nbytes = se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, view.num_units, max_len,
                                       view.struct.max_pages, q_per_kv, view.struct.head_dim, 0)
        return torch.zeros(max(nbytes, 1), dtype=torch.uint8, device=device)

    def attend(self, q, k_new, v_new, new_pos, out, lse=None, accumulate=True, max_len=None):
        """``max_len`` bounds this step's resident slots after the append (the
        scheduler knows it); it sizes the launch.  Defaults to the capacity."""
        se.se_decode_attend(self.view, self.G, q, k_new, v_new, new_pos, None, 0, self.scale,
                            max_len or self.max_len, se.SE_ATTEND_ACCUMULATE if accumulate else 0,
                            out, lse, None, 0, self.ws, self.dev_err)

    def evict(self, max_len=None):
        se.se_evict_compact(self.view, self.budget, self.recent, max_len or self.max_len, self.freed,
                            0 if self.freed is None else self.freed.shape[1], self.freed_count,
                            self.dev_err)

    def step(self, q, k_new, v_new, new_pos, out, lse=None, max_len=None, fused=True):
        """One decode step.  fused: se_decode_step_h2o (attention, score update
        and eviction in one call); otherwise se_decode_attend then se_evict_compact."""
        if fused:
            se.se_decode_step_h2o(self.view, self.G, q, k_new, v_new, new_pos, self.scale, self.budget,
                                  self.recent, max_len or self.max_len, out, lse, self.freed,
                                  0 if self.freed is None else self.freed.shape[1], self.freed_count,
                                  self.ws, self.dev_err)
        else:
            self.attend(q, k_new, v_new, new_pos, out, lse, max_len=max_len)
            self.evict(max_len)


class QuestDecoder:
    """One layer's Quest decode step: page selection (se_quest_select), then
    append + attention over the selected pages and the current page
    (se_decode_attend); step() does both in one call (se_decode_step_quest)."""

    def __init__(self, view: se.KVView, q_per_kv: int, scale: float, top_k: int, max_len: int,
                 device):
        self.view, self.G, self.scale, self.top_k, self.max_len = view, q_per_kv, scale, top_k, max_len
        d = view.struct.head_dim
        mp = view.struct.max_pages
        na = se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, view.num_units, max_len, mp, q_per_kv, d, top_k)
        nq = se.se_workspace_bytes(se.SE_OP_QUEST_SELECT, view.num_units, max_len, mp, q_per_kv, d, 0)
        ns = se.se_workspace_bytes(se.SE_OP_QUEST_STEP, view.num_units, max_len, mp, q_per_kv, d, top_k)
        self.ws_attend = torch.zeros(max(na, ns, 1), dtype=torch.uint8, device=device)
        self.ws_select = torch.zeros(max(nq, 1), dtype=torch.uint8, device=device)
        self.sel = torch.full((view.num_units, top_k), -1, dtype=torch.int32, device=device)
        self.dev_err = torch.zeros(1, dtype=torch.int32, device=device)

    def summarize(self):
        se.se_quest_summarize(self.view, self.max_len, self.dev_err)

    def select(self, q, page_scores=None):
        se.se_quest_select(self.view, self.G, q, self.scale, self.top_k, self.max_len, 0, self.sel,
                           page_scores, 0 if page_scores is None else page_scores.shape[1],
                           self.ws_select, self.dev_err)

    def attend(self, q, k_new, v_new, new_pos, out, lse=None, max_len=None):
        se.se_decode_attend(self.view, self.G, q, k_new, v_new, new_pos, self.sel, self.top_k,
                            self.scale, max_len or self.max_len, 0, out, lse, None, 0,
                            self.ws_attend, self.dev_err)

    def step(self, q, k_new, v_new, new_pos, out, lse=None, max_len=None, fused=True):
        """Selection then attention: in one call (fused), else the two calls."""
        if not fused:
            self.select(q)
            self.attend(q, k_new, v_new, new_pos, out, lse, max_len=max_len)
            return
        se.se_decode_step_quest(self.view, self.G, q, k_new, v_new, new_pos, self.scale, self.top_k,
                                max_len or self.max_len, self.sel, out, lse, self.ws_attend, self.dev_err)


class OmniKVDecoder:
    """A model's OmniKV decode step, layer by layer (Appendix A.3, OmniKV): an
    observation layer appends, attends over every slot keeping the logits
    (se_decode_attend) and selects the b slots with the largest logit over the
    request's heads (se_omnikv_select); each later layer, until the next
    observation layer, appends and attends over that selection of its own cache
    (se_attend_slots).  The selection and the buffers are shared by the layers,
    whose calls run one after another on one stream."""

    def __init__(self, q_per_kv: int, scale: float, budget: int, observation_layers, num_units: int,
                 num_kv_heads: int, max_len: int, max_pages: int, head_dim: int, device):
        self.G, self.scale, self.budget, self.max_len = q_per_kv, scale, budget, max_len
        self.observe = set(int(l) for l in observation_layers)
        num_req = num_units // num_kv_heads
        self.stride = -(-max_len // 64) * 64
        self.logits = torch.empty(num_units * q_per_kv * self.stride, dtype=torch.float32, device=device)
        self.sel = torch.full((num_req, budget), -1, dtype=torch.int32, device=device)
        na = se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, num_units, max_len, max_pages, q_per_kv, head_dim, 0)
        ns = se.se_workspace_bytes(se.SE_OP_OMNIKV_SELECT, num_req, max_len, max_pages, q_per_kv, head_dim, 0)
        self.ws_attend = torch.empty(max(na, 1), dtype=torch.uint8, device=device)
        self.ws_select = torch.empty(max(ns, 1), dtype=torch.uint8, device=device)
        self.dev_err = torch.zeros(1, dtype=torch.int32, device=device)
        self.selected = False

    def layer(self, l: int, view: se.KVView, q, k_new, v_new, new_pos, out, lse=None, max_len=None):
        """Layer l's step.  ``max_len`` bounds the slots after this step's append
        (defaults to the capacity).  The first layer of a step must be an
        observation layer, so that the sparse layers read this step's selection."""
        ml = max_len or self.max_len
        if l in self.observe:
            se.se_decode_attend(view, self.G, q, k_new, v_new, new_pos, None, 0, self.scale, ml, 0, out, lse,
                                self.logits, self.stride, self.ws_attend, self.dev_err)
            se.se_omnikv_select(view, self.G, self.logits, self.stride, self.budget, ml, self.sel,
                                self.ws_select, self.dev_err)
            self.selected = True
        else:
            if not self.selected:
                raise RuntimeError("OmniKV: a sparse layer before any observation layer has selected")
            se.se_attend_slots(view, self.G, q, k_new, v_new, new_pos, self.sel, self.budget, self.scale, ml,
                               out, lse, self.dev_err)
