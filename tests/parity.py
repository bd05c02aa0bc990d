"""Comparison of a GPU routing result with the fp64 oracle.

Rules (written against the selection and gate definitions of the router):
* A token is *excluded* from index-set parity when its oracle k-th and (k+1)-th logits are
  a near tie: |l_(k) - l_(k+1)| < 1e-3 * max(|l_(k)|, |l_(k+1)|).  With k == M there is no
  (k+1)-th logit and nothing is excluded.  Excluded tokens are counted and their set match
  is reported, not asserted.
* For every other token the selected expert *sets* must be identical.
* Gates are compared per expert id: |gate_gpu - gate_oracle| <= 2e-3 (bf16 inputs, fp32
  accumulation), for non-excluded tokens.
* Validity holds for every token: ids in [0, M), no repeats, GPU gates sum to 1 within
  1e-5, and gates are non-increasing in the GPU's selection order.
"""
from __future__ import annotations

import dataclasses

import numpy as np

GATE_TOL = 2e-3
BAND_REL = 1e-3
GATE_SUM_TOL = 1e-5


@dataclasses.dataclass
class ParityReport:
    n: int
    excluded: int
    mismatched: int  # non-excluded tokens whose expert set differs
    excluded_mismatched: int  # excluded tokens whose set differs (reported only)
    max_gate_err: float  # over non-excluded tokens
    mismatch_rows: np.ndarray

    def ok(self) -> bool:
        return self.mismatched == 0 and self.max_gate_err <= GATE_TOL

    def __str__(self):
        return ("tokens=%d excluded(near-tie)=%d mismatched=%d excluded_mismatched=%d "
                "max_gate_err=%.3g" % (self.n, self.excluded, self.mismatched,
                                       self.excluded_mismatched, self.max_gate_err))


def near_tie(orc, k: int, M: int) -> np.ndarray:
    if k >= M:
        return np.zeros(orc.idx.shape[0], dtype=bool)
    a, b = orc.kth, orc.next
    return np.abs(a - b) < BAND_REL * np.maximum(np.abs(a), np.abs(b))


def check_valid(idx: np.ndarray, gate: np.ndarray, M: int):
    assert idx.dtype == np.int32 and gate.dtype == np.float32
    assert np.all((idx >= 0) & (idx < M)), "expert id out of range"
    s = np.sort(idx, axis=1)
    assert np.all(s[:, 1:] != s[:, :-1]), "an expert was selected twice for one token"
    assert np.all(np.isfinite(gate))
    assert np.all(np.abs(gate.astype(np.float64).sum(axis=1) - 1.0) <= GATE_SUM_TOL)
    assert np.all(np.diff(gate, axis=1) <= 1e-7), "gates not in selection order"


def compare(orc, idx: np.ndarray, gate: np.ndarray, k: int, M: int) -> ParityReport:
    """orc: oracle.OracleResult for the same rows as idx/gate (GPU outputs as numpy)."""
    idx = np.asarray(idx)
    gate = np.asarray(gate)
    check_valid(idx, gate, M)
    n = idx.shape[0]
    excl = near_tie(orc, k, M)
    o_sorted = np.sort(orc.idx, axis=1)
    g_order = np.argsort(idx, axis=1, kind="stable")
    g_sorted = np.take_along_axis(idx, g_order, axis=1)
    same = np.all(o_sorted == g_sorted, axis=1)
    o_order = np.argsort(orc.idx, axis=1, kind="stable")
    og = np.take_along_axis(orc.gate, o_order, axis=1)
    gg = np.take_along_axis(gate.astype(np.float64), g_order, axis=1)
    err = np.abs(og - gg).max(axis=1)
    checked = same & ~excl
    mism = ~same & ~excl
    return ParityReport(n=n, excluded=int(excl.sum()), mismatched=int(mism.sum()),
                        excluded_mismatched=int((~same & excl).sum()),
                        max_gate_err=float(err[checked].max()) if checked.any() else 0.0,
                        mismatch_rows=np.nonzero(mism)[0])
