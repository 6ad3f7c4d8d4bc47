"""Test-side glue between the generator's tensors, the oracle and GPU results.

Reads generator output (before any library call touches it) into oracle
states, reads the library's results back in slot order, and holds the parity
tolerances.  Nothing here computes any part of the method.
"""

import numpy as np
import torch

from oracle.state import new_unit
from workloads import unit_slots

# Parity bars.  The arithmetic errs far less than these (fp32 sums of exact
# bf16 products: ~1e-6 relative logits; v_exp_f32 within 1 ulp: ~1e-6
# relative weights).
OUT_ATOL = 1e-2          # attention output, absolute
LSE_ATOL = 1e-3          # log-sum-exp, absolute
U_RTOL = 1e-3            # accumulated scores, relative ...
U_ATOL = 1e-7            # ... with this floor for scores below 1e-4
QUEST_RTOL = 1e-3        # Quest page scores, relative to max(1, |score|)
NEAR_TIE = 1e-4          # a selection may differ only between scores this close (relative)
# The H2O step keeps its per-slot weights as fp16 while they wait for the score
# update (each weight rounded by at most 2^-11 relative, so each new score by
# at most 2^-11 of itself): a float64 retention may swap slots whose scores lie
# within twice the score tolerance of each other.
H2O_NEAR_TIE = 2 * U_RTOL


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().to(torch.float64).numpy()


def oracle_unit(state, unit_row: int):
    """The oracle's view of one unit of generator output (slot order)."""
    K, V, pos, u = unit_slots(state, unit_row)
    return new_unit(f64(K), f64(V), pos.numpy().astype(np.int64),
                    None if u is None else f64(u))


def gpu_unit(state, unit_row: int, length=None):
    """One unit of the library's state, in slot order, as NumPy (K, V bf16 bits too)."""
    K, V, pos, u = unit_slots(state, unit_row, length)
    return {"K": f64(K), "V": f64(V), "Kbits": K.view(torch.int16).numpy(),
            "Vbits": V.view(torch.int16).numpy(), "pos": pos.numpy().astype(np.int64),
            "u": None if u is None else u.numpy().astype(np.float64)}


def assert_scores_close(got, want, what=""):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    tol = np.where(np.abs(want) < 1e-4, U_ATOL, U_RTOL * np.abs(want))
    bad = np.abs(got - want) > tol
    assert not bad.any(), f"{what}: {int(bad.sum())} scores off, worst {np.abs(got - want)[bad].max():.3e}"


def h2o_near_tie(oracle_u_by_pos: dict, kept_gpu: set, kept_oracle: set, tol: float = NEAR_TIE) -> bool:
    """True when the two retained sets differ only by swaps of entries whose
    oracle scores agree to tol, relative (a valid TopK up to the rounding of
    the scores: NEAR_TIE for fp32 arithmetic, H2O_NEAR_TIE for decode-step
    scores)."""
    only_g = kept_gpu - kept_oracle
    only_o = kept_oracle - kept_gpu
    if len(only_g) != len(only_o):
        return False
    for x in only_g:
        for y in only_o:
            ux, uy = oracle_u_by_pos[x], oracle_u_by_pos[y]
            if uy - ux > tol * max(abs(ux), abs(uy)):
                return False
    return True


def quest_near_tie(scores: np.ndarray, sel_gpu, sel_oracle) -> bool:
    """True when the two page selections differ only between pages whose oracle
    scores agree to NEAR_TIE."""
    only_g = set(int(b) for b in sel_gpu) - set(int(b) for b in sel_oracle)
    only_o = set(int(b) for b in sel_oracle) - set(int(b) for b in sel_gpu)
    if len(only_g) != len(only_o):
        return False
    for x in only_g:
        for y in only_o:
            if scores[y] - scores[x] > NEAR_TIE * max(1.0, abs(scores[x]), abs(scores[y])):
                return False
    return True
