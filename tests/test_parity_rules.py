"""The parity rules (oracle/parity.py) on the CPU: the oracle's own result passes, and results
with a planted mistake (a wrong expert, an out-of-band pick on a near tie, drifted gates or
logits, a bad order) are caught by the rule meant for them."""
import numpy as np
import pytest

import oracle
from oracle import parity
from paper_2609_36301_amd.inputs import make_inputs

K = 6


@pytest.fixture(scope="module")
def case():
    # duplicated expert columns give exact logit ties, so some tokens sit on a near tie
    inp = make_inputs(400, 64, 16, 120, seed=17, dup_expert_frac=0.2)
    orc = oracle.route_lowrank(inp.x, inp.R1, inp.R2, K)
    full = oracle.route_lowrank(inp.x, inp.R1, inp.R2, inp.R2.shape[1])  # every expert ranked
    return inp, orc, full


def result_of(orc):
    return (orc.idx.copy(), orc.gate.astype(np.float32), orc.topval.astype(np.float32))


def report(inp, idx, gate, topval):
    return parity.evaluate(inp.x, inp.R1, inp.R2, K, idx, gate, topval)


def test_oracle_result_passes(case):
    inp, orc, _ = case
    rep = report(inp, *result_of(orc))
    assert rep.ok(), str(rep)
    assert rep.mismatched == 0 and rep.band_violations == 0 and rep.excluded_mismatched == 0
    assert rep.excluded > 0  # the tie case is exercised


def _clear_token(orc, full):
    excl = parity.near_tie(orc, K, full.idx.shape[1])
    gap = full.topval[:, K - 1] - full.topval[:, K + 3]
    return int(np.nonzero(~excl & (gap > 0.05))[0][0])


def test_wrong_expert_is_a_mismatch_and_a_band_violation(case):
    inp, orc, full = case
    idx, gate, topval = result_of(orc)
    t = _clear_token(orc, full)
    idx[t, K - 1] = full.idx[t, K + 3]  # a clearly worse expert replaces the k-th
    topval[t, K - 1] = full.topval[t, K + 3]
    rep = report(inp, idx, gate, topval)
    assert rep.mismatched == 1 and rep.band_violations == 1 and not rep.ok()
    assert list(rep.mismatch_rows) == [t]


def test_near_tie_swap_is_allowed_but_a_far_pick_is_not(case):
    inp, orc, full = case
    excl = np.nonzero(parity.near_tie(orc, K, full.idx.shape[1]))[0]
    t = int(excl[0])
    idx, gate, topval = result_of(orc)
    # the k-th and (k+1)-th are tied: picking the (k+1)-th is a valid top k
    idx[t, K - 1] = full.idx[t, K]
    topval[t, K - 1] = full.topval[t, K]
    order = np.lexsort((idx[t], -topval[t].astype(np.float64)))
    idx[t], topval[t] = idx[t][order], topval[t][order]
    rep = report(inp, idx, gate, topval)
    assert rep.excluded_mismatched == 1 and rep.band_violations == 0 and rep.ok(), str(rep)
    # a pick far below the boundary is not
    far = int(np.nonzero(full.topval[t] < full.topval[t, K - 1] - 0.2)[0][0])
    idx2, gate2, topval2 = result_of(orc)
    idx2[t, K - 1] = full.idx[t, far]
    topval2[t, K - 1] = full.topval[t, far]
    rep2 = report(inp, idx2, gate2, topval2)
    assert rep2.band_violations == 1 and not rep2.ok()


def test_gate_drift_is_caught(case):
    inp, orc, _ = case
    idx, gate, topval = result_of(orc)
    gate[3, 0] += 3e-3
    gate[3, 1] -= 3e-3
    rep = report(inp, idx, gate, topval)
    assert rep.max_gate_err > parity.GATE_TOL and not rep.ok()


def test_topval_drift_is_caught(case):
    inp, orc, _ = case
    idx, gate, topval = result_of(orc)
    topval[5, K - 1] -= 1e-3 * (1 + abs(topval[5, K - 1]))
    rep = report(inp, idx, gate, topval)
    assert rep.max_topval_err > parity.TOPVAL_REL and not rep.ok()


def test_invalid_rows_are_refused(case):
    inp, orc, _ = case
    idx, gate, topval = result_of(orc)
    bad = idx.copy()
    bad[0, 1] = bad[0, 0]
    with pytest.raises(AssertionError):
        report(inp, bad, gate, topval)
    swapped = idx.copy()
    swapped[1, [0, 1]] = swapped[1, [1, 0]]  # ids out of logit order
    tv = topval.copy()
    with pytest.raises(AssertionError):
        report(inp, swapped, gate, tv[:, ::-1].copy())
    g = gate.copy()
    g[2] *= 1.01  # no longer sums to one
    with pytest.raises(AssertionError):
        report(inp, idx, g, topval)


def test_rows_subset_matches_full_report(case):
    inp, orc, _ = case
    idx, gate, topval = result_of(orc)
    rows = np.arange(0, 400, 7)
    rep = parity.evaluate(inp.x, inp.R1, inp.R2, K, idx, gate, topval, rows=rows)
    assert rep.n == rows.size and rep.ok()
