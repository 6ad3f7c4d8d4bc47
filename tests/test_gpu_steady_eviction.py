"""The fused steady-state H2O step (se_decode_step_h2o) at the launch shapes the
benchmark times, with exact score ties injected, against the oracle.

In steady state a unit holds B slots, appends one and evicts one (Appendix
A.3, eq. background-h2o-retention with |A| = B + 1).  The benchmark passes the
step's bound max_len = B + 1, so one work-group streams each unit and the
eviction runs in the attention kernel's epilogue.  Which epilogue runs
depends on the launch:

  units  B     window  threads  path
  -----  ----  ------  -------  ---------------------------------------------
   512   128    16      512     finish_steady (rows kept per wavefront)
    16   128    16     1024     finish_steady
   256  2048   256     1024     finish_steady
   512  2048   256      512     finish_steady: the 8B layer's steady launch
   512  4096   512      512     finish_steady_strided: the ragged batch's and
                                the 32-layer loop's steady launch
   256  4096   512     1024     finish_steady_strided
   256  8192   512     1024     general retention in the epilogue (B + 1 is
                                past the register-resident steady case)
   512  2048   256      512     general retention in the epilogue: recent
        (gapped positions)      positions that are not one contiguous run

Groups of 8 query heads per KV head repeat four of them: 512 x 2048 takes
finish_steady with fp16 weights, 512 x 4096 the strided one, 16 x 2048 the
1024-thread finish_steady (its 129 pages fit the fp16 weight buffer), 256 x
8192 the general retention.

Ties: six slots of one page, all outside the recent window for the whole run,
get the same key (zero), the same value row and the same score (zero); every
other slot starts at 0.5 or more.  Their accumulated scores stay bit-equal (one
wavefront computes a page's weights) and lowest, so each step must evict the
tied slot with the largest position (larger score first, then lower position,
is the retention order).  The protocol in tests/protocol.py compares every
unit at every step with the oracle fed the GPU's own fp32 scores.
"""
import numpy as np
import pytest
import torch

from tests.protocol import PAGE, h2o_trajectory, read_units
from workloads import StepInputs, isolated_units, scaled, to_device

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
D, HKV = 128, 8
N_STEPS = 4
N_TIE = 6


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _tied_state(units, budget, recent, mode, seed):
    """units of B resident slots (positions per ``mode``), scores >= 0.5 except
    a tie group of N_TIE slots in one page with key 0, one shared value row
    and score 0, whose positions stay outside the window for N_STEPS steps."""
    max_pages = -(-(budget + 1) // PAGE)
    host = isolated_units([budget] * units, max_pages, D, seed=seed, num_kv_heads=HKV, position_mode=mode,
                          score_levels=64)
    g = torch.Generator().manual_seed(seed + 1)
    tie_pos = []
    for u in range(units):
        bt = host.block_table[u].to(torch.int64)
        s = torch.arange(budget)
        ph, row = bt[s // PAGE], s % PAGE
        pos = host.pos_pool[ph, row].to(torch.int64)
        cut = torch.sort(pos, descending=True).values[recent + N_STEPS + 1]
        host.score_pool[ph, row] = 0.5 + 0.5 * host.score_pool[ph, row]
        # a page with at least N_TIE slots below the window's reach
        for page in torch.randperm(budget // PAGE, generator=g).tolist():
            rows = [r for r in range(PAGE) if int(pos[page * PAGE + r]) < int(cut)]
            if len(rows) >= N_TIE:
                break
        rows = rows[:N_TIE]
        p = int(bt[page])
        host.kv_pool[p, 0, rows] = 0
        host.kv_pool[p, 1, rows] = host.kv_pool[p, 1, rows[0]].clone()
        host.score_pool[p, rows] = 0.0
        tie_pos.append(sorted(int(pos[page * PAGE + r]) for r in rows))
    return host, tie_pos


def _steps(num_req, start_pos, seed, G):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((N_STEPS, 1, num_req, HKV * G, D), generator=g).to(torch.bfloat16)
    k = torch.randn((N_STEPS, 1, num_req, HKV, D), generator=g).to(torch.bfloat16)
    v = torch.randn((N_STEPS, 1, num_req, HKV, D), generator=g).to(torch.bfloat16)
    p = (torch.tensor(start_pos, dtype=torch.int64)[None, :] + torch.arange(N_STEPS)[:, None]).to(torch.int32)
    return StepInputs(q=q.to(DEV), k_new=k.to(DEV), v_new=v.to(DEV), new_pos=p.to(DEV))


CASES = [
    # units, budget, window, positions, query heads per KV head
    (512, 128, 16, "permuted", 4),
    (16, 128, 16, "permuted", 4),
    (256, 2048, 256, "permuted", 4),
    (512, 2048, 256, "permuted", 4),
    (512, 4096, 512, "permuted", 4),
    (256, 4096, 512, "permuted", 4),
    (256, 8192, 512, "permuted", 4),
    (512, 2048, 256, "gapped", 4),
    # groups of 8: per-wavefront rows (fp16 weights), strided, wide, general
    (512, 2048, 256, "permuted", 8),
    (512, 4096, 512, "permuted", 8),
    (16, 2048, 256, "permuted", 8),
    (256, 8192, 512, "permuted", 8),
]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("units,budget,recent,mode,G", CASES)
def test_steady_step_with_ties(se, units, budget, recent, mode, G):
    seed = units + budget + recent + len(mode) + (G - 4)
    print(f"case units={units} B={budget} w={recent} {mode} G={G}", flush=True)
    host, tie_pos = _tied_state(units, budget, recent, mode, seed)
    gs = to_device(host, DEV)
    gs.w = scaled(gs.w, hq=HKV * G, hkv=HKV, num_req=units // HKV)
    num_req = units // HKV
    # new positions continue above every resident one (per request: its units share them)
    top = host.pos_pool.max().item() + 1
    steps = _steps(num_req, [top] * num_req, seed + 2, G)
    bounds = [budget + 1] * N_STEPS  # the benchmark's steady bound
    checked, near = h2o_trajectory(se, gs, steps, N_STEPS, {0: range(units)}, q_per_kv=G, scale=float(np.float32(D ** -0.5)),
                                   budget=budget, recent=recent, bounds=bounds, device=DEV)
    assert checked == N_STEPS * units
    # each step evicted the tied slot with the largest position
    final = read_units(gs, range(units), with_kv=False)
    for u in range(units):
        left = set(final[u]["pos"].tolist())
        tp = tie_pos[u]
        assert all(p in left for p in tp[:N_TIE - N_STEPS]), (u, tp)
        assert not any(p in left for p in tp[N_TIE - N_STEPS:]), (u, tp)
