"""The seeded input generator (variance lemma of the initialization appendix, recipes)."""
import math

import numpy as np

from paper_2609_36301_amd.inputs import (WORKLOADS, bf16_bits_to_f32, f32_to_bf16_bits,
                                         make_inputs, make_workload_inputs, transposed_factors)


def test_bf16_rounding_round_trip_and_ties():
    vals = np.array([1.0, -2.5, 3.140625, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 65504.0], np.float32)
    b = f32_to_bf16_bits(vals)
    back = bf16_bits_to_f32(b)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: ties go to the even mantissa (1.0)
    assert back[3] == 1.0
    assert back[4] == 1.0 + 2**-6
    assert back[0] == 1.0 and back[1] == -2.5
    # every bf16 value survives a round trip
    allbits = np.arange(0, 0x7F80, 7, dtype=np.uint16)
    assert np.array_equal(f32_to_bf16_bits(bf16_bits_to_f32(allbits)), allbits)


def test_seeded_reproducible():
    a = make_inputs(64, 128, 16, 200, seed=3)
    b = make_inputs(64, 128, 16, 200, seed=3)
    c = make_inputs(64, 128, 16, 200, seed=4)
    assert np.array_equal(a.x, b.x) and np.array_equal(a.R2, b.R2)
    assert not np.array_equal(a.x, c.x)


def test_variance_lemma():
    """Var(z_i) = |x|^2/h ~ 1 and Var(l_e) = r * (1/h) * (1/r) * |x|^2 ~ 1 (within 3%)."""
    inp = make_inputs(2048, 512, 32, 1024, seed=0)
    x = bf16_bits_to_f32(inp.x).astype(np.float64)
    z = x @ bf16_bits_to_f32(inp.R1).astype(np.float64)
    logit = z @ bf16_bits_to_f32(inp.R2).astype(np.float64)
    assert abs(z.var() - 1.0) < 0.03, z.var()
    assert abs(logit.var() - 1.0) < 0.03, logit.var()
    assert abs(x.var() - 1.0) < 0.01


def test_duplicate_tokens_bit_identical():
    inp = make_inputs(1000, 64, 16, 32, seed=1, dup_token_frac=0.05)
    assert inp.dup_dst.size == 50
    assert len(set(inp.dup_dst.tolist())) == 50
    assert not set(inp.dup_src.tolist()) & set(inp.dup_dst.tolist())
    assert np.array_equal(inp.x[inp.dup_dst], inp.x[inp.dup_src])


def test_expert_bias_is_per_column():
    base = make_inputs(16, 64, 16, 4000, seed=2)
    biased = make_inputs(16, 64, 16, 4000, seed=2, expert_bias_var=0.5)
    shift = (bf16_bits_to_f32(biased.R2).astype(np.float64)
             - bf16_bits_to_f32(base.R2).astype(np.float64))
    col_mean = shift.mean(axis=0)
    # the offset is shared by the column (up to bf16 rounding) and has variance 0.5
    assert np.all(np.abs(shift - col_mean[None, :]) <= 0.02 * (1 + np.abs(col_mean[None, :])))
    assert abs(col_mean.var() - 0.5) < 0.05


def test_duplicate_experts_make_exact_ties():
    inp = make_inputs(8, 32, 16, 100, seed=5, dup_expert_frac=0.05)
    cols = {tuple(inp.R2[:, e]) for e in range(100)}
    assert len(cols) == 95


def test_workloads_and_layouts():
    assert set(WORKLOADS) == {"tiny", "teaser_prefill", "mid", "fine_grained", "decode"}
    w = WORKLOADS["tiny"]
    inp = make_workload_inputs("tiny")
    assert inp.shape == (w.T, w.h, w.r, w.M)
    r1t, r2t = transposed_factors(inp)
    assert r1t.shape == (w.r, w.h) and r2t.shape == (w.M, w.r)
    assert np.array_equal(r1t.T, inp.R1) and np.array_equal(r2t.T, inp.R2)
    small = make_workload_inputs("mid", T=400)
    assert small.shape == (400, 2048, 64, 16384) and small.dup_dst.size == 20
    assert math.isclose(WORKLOADS["fine_grained"].expert_bias_var, 0.5)
