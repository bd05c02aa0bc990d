"""Comparison of a routing result with the fp64 oracle (test infrastructure).

TEST INFRASTRUCTURE ONLY, like the rest of this package: the test suite, the smoke check and
the benchmark's CPU-baseline leg are its only callers.

Rules, written against the selection and gate definitions of the router ("Preliminaries",
softmax over the TopK of the logits):

* Near ties.  A token is *excluded* from index-set parity when its oracle k-th and (k+1)-th
  logits differ by less than 1e-3 relative: |l_(k) - l_(k+1)| < 1e-3 max(|l_(k)|, |l_(k+1)|).
  With k == M there is no (k+1)-th logit and nothing is excluded.
* Every other token: the selected expert *set* must equal the oracle's.
* Every token, excluded or not, must hold a *band-valid* top k: with l the oracle's fp64
  logits, the smallest logit of the selected experts may fall short of the largest logit of
  the unselected experts by at most 1e-3 relative.  The unselected maximum is exact: it is
  the best oracle-selected expert the result left out, or l_(k+1) when it left none out.
  The logits of the result's own picks come from oracle.logits_at.
* Gates, per expert id, on every expert the result shares with the oracle (all k experts
  for non-excluded tokens): |gate - gate_oracle| <= 2e-3.  Excluded tokens are held to the
  same bound on their shared experts and reported separately.
* Selected logits (when given): |topval - l| <= 1e-4 (1 + |l|) for every pick, against the
  oracle logit of that very expert.
* Validity of every row: ids in [0, M), no repeats, gates finite, summing to 1 within 1e-5
  and non-increasing in selection order; with topval, the order is logit descending, ties by
  smaller id.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from . import logits_at, route_lowrank

GATE_TOL = 2e-3
BAND_REL = 1e-3
GATE_SUM_TOL = 1e-5
TOPVAL_REL = 1e-4


@dataclasses.dataclass
class ParityReport:
    n: int
    excluded: int  # near-tie tokens (oracle k-th and (k+1)-th within 1e-3 relative)
    mismatched: int  # non-excluded tokens whose expert set differs from the oracle's
    excluded_mismatched: int  # excluded tokens whose set differs (must still be band-valid)
    band_violations: int  # tokens whose selection is not a band-valid top k
    max_gate_err: float  # over the experts of non-excluded tokens
    max_gate_err_excluded: float  # over the shared experts of excluded tokens
    max_topval_err: float  # max |topval - l| / (1 + |l|) over every pick (0 without topval)
    mismatch_rows: np.ndarray  # positions (in the compared rows) of mismatched tokens
    band_rows: np.ndarray  # positions of band-violating tokens

    def ok(self) -> bool:
        return (self.mismatched == 0 and self.band_violations == 0
                and self.max_gate_err <= GATE_TOL and self.max_gate_err_excluded <= GATE_TOL
                and self.max_topval_err <= TOPVAL_REL)

    def as_dict(self) -> dict:
        return {"tokens": self.n, "excluded": self.excluded, "mismatched": self.mismatched,
                "excluded_mismatched": self.excluded_mismatched,
                "band_violations": self.band_violations,
                "max_gate_err": float("%.3g" % self.max_gate_err),
                "max_gate_err_excluded": float("%.3g" % self.max_gate_err_excluded),
                "max_topval_rel_err": float("%.3g" % self.max_topval_err),
                "ok": self.ok()}

    def __str__(self):
        return ("tokens=%d excluded(near-tie)=%d mismatched=%d excluded_mismatched=%d "
                "band_violations=%d max_gate_err=%.3g max_gate_err_excluded=%.3g "
                "max_topval_err=%.3g" % (self.n, self.excluded, self.mismatched,
                                         self.excluded_mismatched, self.band_violations,
                                         self.max_gate_err, self.max_gate_err_excluded,
                                         self.max_topval_err))


def near_tie(orc, k: int, M: int) -> np.ndarray:
    if k >= M:
        return np.zeros(orc.idx.shape[0], dtype=bool)
    a, b = orc.kth, orc.next
    return np.abs(a - b) < BAND_REL * np.maximum(np.abs(a), np.abs(b))


def check_valid(idx: np.ndarray, gate: np.ndarray, M: int, topval=None):
    assert idx.dtype == np.int32 and gate.dtype == np.float32
    assert np.all((idx >= 0) & (idx < M)), "expert id out of range"
    s = np.sort(idx, axis=1)
    assert np.all(s[:, 1:] != s[:, :-1]), "an expert was selected twice for one token"
    assert np.all(np.isfinite(gate))
    assert np.all(np.abs(gate.astype(np.float64).sum(axis=1) - 1.0) <= GATE_SUM_TOL)
    assert np.all(np.diff(gate, axis=1) <= 1e-7), "gates not in selection order"
    if topval is not None:
        a, b = topval[:, :-1], topval[:, 1:]
        ordered = (a > b) | ((a == b) & (idx[:, :-1] < idx[:, 1:]))
        assert np.all(ordered), "selection not in (logit descending, id ascending) order"


def compare(orc, idx: np.ndarray, gate: np.ndarray, k: int, M: int, picked_logits: np.ndarray,
            topval=None) -> ParityReport:
    """orc: oracle result for the compared rows; idx/gate/topval: the result on the same rows;
    picked_logits: oracle logits at the result's picks (oracle.logits_at(rows, idx))."""
    idx = np.asarray(idx)
    gate = np.asarray(gate)
    check_valid(idx, gate, M, topval)
    n = idx.shape[0]
    excl = near_tie(orc, k, M)
    # membership of each oracle pick in the result's set, and vice versa
    o_in_g = (orc.idx[:, :, None] == idx[:, None, :]).any(axis=2)  # [n][k]
    same = o_in_g.all(axis=1)
    # band validity: min over picks >= max over unselected - band (exact unselected max)
    min_sel = picked_logits.min(axis=1)
    left_out = np.where(o_in_g, -np.inf, orc.topval).max(axis=1)
    max_unsel = np.maximum(left_out, orc.next) if k < M else left_out
    band = BAND_REL * np.maximum(np.abs(min_sel), np.abs(max_unsel))
    bad_band = (min_sel < max_unsel - band) & np.isfinite(max_unsel)
    # gates on shared experts, matched by id
    g_of = np.where(orc.idx[:, :, None] == idx[:, None, :], gate[:, None, :].astype(np.float64),
                    0.0).sum(axis=2)  # result's gate of each oracle pick (0 if not picked)
    gerr = np.where(o_in_g, np.abs(g_of - orc.gate), 0.0).max(axis=1)
    checked = same & ~excl
    mism = ~same & ~excl
    terr = 0.0
    if topval is not None:
        terr = float((np.abs(topval.astype(np.float64) - picked_logits) /
                      (1.0 + np.abs(picked_logits))).max()) if n else 0.0
    return ParityReport(
        n=n, excluded=int(excl.sum()), mismatched=int(mism.sum()),
        excluded_mismatched=int((~same & excl).sum()), band_violations=int(bad_band.sum()),
        max_gate_err=float(gerr[checked].max()) if checked.any() else 0.0,
        max_gate_err_excluded=float(gerr[excl].max()) if excl.any() else 0.0,
        max_topval_err=terr, mismatch_rows=np.nonzero(mism)[0], band_rows=np.nonzero(bad_band)[0])


def evaluate(x, R1, R2, k: int, idx, gate, topval=None, rows=None, threads=None) -> ParityReport:
    """Runs the oracle on the rows (all tokens when rows is None) of the bf16 inputs x [T][h],
    R1 [h][r], R2 [r][M] and compares the result idx/gate/topval ([T][k], all tokens) with it."""
    T = x.shape[0]
    M = R2.shape[1]
    orc = route_lowrank(x, R1, R2, k, rows=rows, threads=threads)
    return compare_with(orc, x, R1, R2, k, idx, gate, topval, rows, threads)


def compare_with(orc, x, R1, R2, k: int, idx, gate, topval=None, rows=None,
                 threads=None) -> ParityReport:
    """As evaluate, with the oracle result for those rows already computed."""
    T = x.shape[0]
    M = R2.shape[1]
    r = np.arange(T, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    sel = np.ascontiguousarray(np.asarray(idx)[r])
    picked = logits_at(x, R1, R2, r, sel, threads=threads)
    tv = None if topval is None else np.asarray(topval)[r]
    return compare(orc, sel, np.asarray(gate)[r], k, M, picked, tv)
