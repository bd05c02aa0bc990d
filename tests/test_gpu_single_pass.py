"""GPU parity of the single-pass route (the library's choice for at least 4096 tokens and at least
32768 experts): oracle parity on every token, agreement with the resident route (m_chunks = 8,
two full sweeps) and the histogram.  The single-pass route computes z = x R1 in its own
summation order, so its fp32 logits can differ from the resident route's in the last bits:
selections agree wherever the k-th and (k+1)-th logits are not within rounding of each other.

Shapes cover every rank width (r = 16, 32, 64), every top-K list size of the kernels (k = 1, 2,
3, 5, 16), ragged token counts (a partial 512-token block and a partial 64-token group) and
ragged expert counts (a partial last tile), plus the degenerate and tied cases that send tokens
down the finalize kernel's exact sweep.
"""
import numpy as np
import pytest

import oracle
from oracle import parity
from gpu_util import route_lowrank
from paper_2609_36301_amd import router
from paper_2609_36301_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu

SHAPES = [
    (4100, 256, 16, 33000, 1),
    (4096, 512, 32, 40000, 5),
    (4500, 128, 64, 32768, 2),
    (4200, 64, 32, 36001, 3),
    (5000, 256, 64, 65600, 16),
]


def _check(inp, k, idx, gate, topval, label):
    rep = parity.evaluate(inp.x, inp.R1, inp.R2, k, idx, gate, topval)
    print("[parity] single-pass %s %s" % (label, rep), flush=True)
    assert rep.ok(), "%s: %s mismatched rows %s band rows %s" % (
        label, rep, rep.mismatch_rows[:10], rep.band_rows[:10])


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_single_pass_parity_and_resident_route_agreement(shape):
    T, h, r, M, k = shape
    assert router.lowrank_route(T, h, r, M, k) == "single-pass"
    inp = make_inputs(T, h, r, M, seed=T + M + k, expert_bias_var=0.25)
    idx, gate, topval, counts = route_lowrank(inp, k, histogram=True, tag="single-pass")
    _check(inp, k, idx, gate, topval, str(shape))
    assert np.array_equal(counts, oracle.histogram(idx, M).astype(np.int32))
    _agree_with_resident(inp, k, idx, topval)


def _agree_with_resident(inp, k, idx, topval):
    ref_idx, _, ref_tv, _ = route_lowrank(inp, k, m_chunks=8, tag="resident")
    same = np.all(idx == ref_idx, axis=1)
    # differing rows: a near tie at the k-th logit (both selections then pass the band check)
    assert same.mean() > 0.999, same.mean()
    assert np.allclose(topval[same], ref_tv[same], rtol=1e-5, atol=1e-6)


def test_single_pass_zero_tokens_take_the_exact_sweep():
    """Zero-vector tokens tie every expert at logit 0: their record lists overflow and the
    finalize kernel sweeps all experts exactly.  Expected: experts 0..k-1, gates 1/k, logits 0."""
    T, h, r, M, k = 4096, 256, 32, 33000, 8
    inp = make_inputs(T, h, r, M, seed=5)
    zero_rows = [0, 63, 64, 511, 512, 2047, 4095]
    inp.x[zero_rows] = 0
    idx, gate, topval, counts = route_lowrank(inp, k, histogram=True, tag="single-pass zero")
    for t in zero_rows:
        assert np.array_equal(idx[t], np.arange(k, dtype=np.int32))
        assert np.allclose(gate[t], 1.0 / k, atol=1e-7)
        assert np.all(topval[t] == 0.0)
    _check(inp, k, idx, gate, topval, "zero tokens")
    assert np.array_equal(counts, oracle.histogram(idx, M).astype(np.int32))


def test_single_pass_exact_ties_resolve_to_lower_expert():
    """Duplicated expert columns give identical logits (and identical screening bounds): the
    lower expert id must win, as in the oracle's order."""
    T, h, r, M, k = 4096, 256, 32, 40000, 8
    inp = make_inputs(T, h, r, M, seed=78, dup_expert_frac=0.05)
    idx, gate, topval, _ = route_lowrank(inp, k, tag="single-pass ties")
    orc = oracle.route_lowrank(inp.x, inp.R1, inp.R2, k)
    rep = parity.compare_with(orc, inp.x, inp.R1, inp.R2, k, idx, gate, topval)
    print("[parity] single-pass ties %s" % rep, flush=True)
    assert rep.ok(), str(rep)
    _agree_with_resident(inp, k, idx, topval)
