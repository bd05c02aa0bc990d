"""GPU parity of the training forward pass (more_route_lowrank_train) against the oracle: the
routing under the routing tests' rules, and the softmax statistics m, Z and psum within the
tolerance derived below (marked `gpu`).

Tolerance.  m is the routing's top-1 logit, held to the routing tests' logit contract
|m - m*| <= 1e-4 (1 + |m*|).  Z and psum take their logits from the matrix cores with z carried
as a bfloat16 hi/lo pair: with A_t = max_e |l_te| and S_t = max_e sum_i |z_ti u_ei|, every
exponent l - m of token t is within
    d_t = 1e-4 (1 + A_t) + 2^-18 S_t + (2r + 1) 2^-24 (A_t + S_t)
of exact (the logit contract for z itself, the hi/lo rounding of z, and the fp32 accumulation of
2r products and the bias).  Then |Z / Z* - 1| <= exp(2 d_t) - 1 plus fp32 summation of at most M
terms, and every probability P_te = exp(l - m - ln Z) is within exp(4 d_t) - 1 relative, so
|psum - psum*| <= sum_t P_te (exp(4 d_t) - 1) plus fp32 summation of at most T terms.  A few ulp
of v_exp_f32 and log2f are added as 1e-6 relative.

A dropped or doubled expert or token moves these sums by far more than the tolerance in the
small cases (a handful of experts or tokens per sum) and in the planted cases (tokens that put
almost all their probability on one expert, placed at expert tile boundaries, in the ragged last
expert tile and in the ragged last token tile).
"""
import numpy as np
import pytest

import oracle
from oracle import parity
from gpu_util import announce, require_gpu, to_dev
from paper_2609_36301_amd.inputs import (WORKLOADS, bf16_bits_to_f32, f32_to_bf16_bits,
                                         make_inputs, make_workload_inputs, transposed_factors)

pytestmark = pytest.mark.gpu


def f64(bits):
    return bf16_bits_to_f32(bits).astype(np.float64)


def _run(inp, k, tag, topval=True, histogram=True):
    torch = require_gpu()
    from paper_2609_36301_amd import router
    T, h, r, M = inp.shape
    R1t, R2t = transposed_factors(inp)
    announce("%s route_lowrank_train T=%d h=%d r=%d M=%d k=%d seed=%d route=%s"
             % (tag, T, h, r, M, k, inp.seed, router.lowrank_route(max(T, 1), h, r, M, k)))
    x_d, r1_d, r2_d = to_dev(inp.x), to_dev(R1t), to_dev(R2t)
    out = router.route_lowrank_train(x_d, r1_d, r2_d, k, topval=topval, histogram=histogram)
    torch.cuda.synchronize()
    res = {name: (None if getattr(out, name) is None else getattr(out, name).cpu().numpy())
           for name in ("idx", "gate", "topval", "counts", "m", "Z", "psum")}
    del x_d, r1_d, r2_d, out
    return res


def _tolerances(inp, m, Z):
    """Per token the exponent bound d_t (A_t = max_e |l_te|, S_t = max_e sum_i |z_ti u_ei|), and
    per expert W_e = sum_t P_te (exp(4 d_t) - 1), from fp64 logits in blocks of 256 tokens."""
    T, h, r, M = inp.shape
    z = f64(inp.x) @ f64(inp.R1)
    R2 = f64(inp.R2)
    aR2 = np.abs(R2)
    d, W = np.zeros(T), np.zeros(M)
    for t0 in range(0, T, 256):
        zz = z[t0:t0 + 256]
        lg = zz @ R2
        A = np.abs(lg).max(axis=1)
        S = (np.abs(zz) @ aR2).max(axis=1)
        dd = 1e-4 * (1 + A) + 2.0 ** -18 * S + (2 * r + 1) * 2.0 ** -24 * (A + S)
        d[t0:t0 + 256] = dd
        P = np.exp(lg - m[t0:t0 + 256, None]) / Z[t0:t0 + 256, None]
        W += np.expm1(4 * dd) @ P
    return d, W


def _check_stats(inp, k, got, tag):
    T, h, r, M = inp.shape
    m, Z, psum = oracle.route_stats(inp.x, inp.R1, inp.R2)
    d, W = _tolerances(inp, m, Z)
    gm, gZ, gp = (got[n].astype(np.float64) for n in ("m", "Z", "psum"))
    assert np.all(np.isfinite(gm)) and np.all(np.isfinite(gZ)) and np.all(np.isfinite(gp))
    # m: the routing's top-1 logit, bit for bit, within the logit contract of the oracle's
    if got["topval"] is not None:
        assert np.array_equal(got["m"], got["topval"][:, 0]), tag
    m_err = np.abs(gm - m) / (1 + np.abs(m))
    assert m_err.max() <= 1e-4, (tag, m_err.max())
    # Z, token by token
    z_tol = np.expm1(2 * d) + 2.0 ** -24 * (M + 64) + 1e-6
    z_err = np.abs(gZ / Z - 1)
    bad = np.nonzero(z_err > z_tol)[0]
    assert bad.size == 0, (tag, "Z", bad[:10], z_err[bad[:10]], z_tol[bad[:10]])
    # psum, expert by expert
    p_tol = W + psum * (2.0 ** -24 * (T + 64) + 1e-6) + 1e-30
    p_abs = np.abs(gp - psum)
    badp = np.nonzero(p_abs > p_tol)[0]
    assert badp.size == 0, (tag, "psum", badp[:10], p_abs[badp[:10]], p_tol[badp[:10]])
    assert abs(gp.sum() - T) <= p_tol.sum() + 1e-3, (tag, gp.sum(), T)
    p_rel = p_abs / np.maximum(psum, 1e-30)
    print("[train] %s T=%d M=%d max m err %.3g; Z: max rel err %.3g, min tol %.3g; psum: max rel "
          "err %.3g, max err/tol %.3g" % (tag, T, M, m_err.max(), z_err.max(), z_tol.min(),
                                          p_rel.max(), (p_abs / p_tol).max()), flush=True)


def _check_routing(inp, k, got, tag, rows=None):
    rep = parity.evaluate(inp.x, inp.R1, inp.R2, k, got["idx"], got["gate"], got["topval"],
                          rows=rows)
    print("[parity] train %s %s" % (tag, rep), flush=True)
    assert rep.ok(), "%s: %s" % (tag, rep)
    if got["counts"] is not None:
        assert np.array_equal(got["counts"], oracle.histogram(got["idx"], inp.shape[3]))


SHAPES = [
    (256, 512, 16, 256, 8),      # one-launch route
    (300, 64, 16, 33, 2),        # ragged tokens, one full tile plus one expert
    (77, 64, 32, 5, 2),          # fewer experts than a tile
    (100, 32, 16, 1, 1),         # one expert: Z = 1, psum = T
    (1000, 256, 32, 5000, 16),   # fused route, k = 16
    (513, 64, 64, 1100, 3),      # fused route, ragged both ways
    (2000, 128, 64, 20000, 8),   # expert-resident route
    (4100, 256, 32, 33000, 4),   # single-pass route
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_train_parity(shape):
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=T + M + k, expert_bias_var=0.25)
    got = _run(inp, k, "parity")
    _check_routing(inp, k, got, str(shape))
    _check_stats(inp, k, got, str(shape))


PLANTED = [
    (1500, 128, 32, 40001, 8),   # expert-resident route; last tile holds one expert
    (4100, 256, 64, 33001, 4),   # single-pass route
    (513, 64, 64, 1100, 3),      # fused route
    (300, 64, 16, 2000, 2),      # one-launch route
]


@pytest.mark.parametrize("shape", PLANTED, ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_train_planted_experts(shape):
    """Up to 64 tokens, the last one (in a partial 32-token tile) among them, each get an expert
    of their own whose row points along the token's z with logit about 16, so that the token puts
    almost all its probability there.  The planted experts sit at both ends of expert tiles, at
    the first and last expert, and spread over the expert axis: a skipped or doubled expert
    tile, expert row or token anywhere near a boundary moves that token's Z or the expert's psum
    by order one."""
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=T + M)
    rng = np.random.default_rng(M)
    z = f64(inp.x) @ f64(inp.R1)
    Mt = (M + 31) // 32
    ends = np.concatenate([32 * np.arange(Mt), np.minimum(32 * np.arange(Mt) + 31, M - 1)])
    pool = np.setdiff1d(np.unique(ends), [0, M - 1])
    n = min(64, T, pool.size + 2)
    toks = np.concatenate([np.sort(rng.choice(T - 1, size=n - 1, replace=False)), [T - 1]])
    experts = np.concatenate([[0], rng.permutation(pool)[:n - 2], [M - 1]])
    assert experts.size == toks.size == n
    R2 = bf16_bits_to_f32(inp.R2).copy()
    for t, e in zip(toks, experts):
        R2[:, e] = (16.0 / (z[t] @ z[t])) * z[t]
    inp.R2 = f32_to_bf16_bits(R2.astype(np.float32))
    got = _run(inp, k, "planted experts")
    # the planted pairs really dominate their tokens
    m, Z, _ = oracle.route_stats(inp.x, inp.R1, inp.R2)
    l_planted = (f64(inp.x[toks]) @ f64(inp.R1) * f64(inp.R2[:, experts]).T).sum(axis=1)
    share = np.exp(l_planted - m[toks]) / Z[toks]
    assert np.median(share) > 0.5, np.median(share)
    _check_routing(inp, k, got, "planted experts")
    _check_stats(inp, k, got, "planted experts")


def test_train_zero_tokens_tie_every_expert():
    T, h, r, M, k = 600, 64, 32, 3000, 4
    inp = make_inputs(T, h, r, M, seed=31)
    zero_rows = [0, 31, 32, 511, 512, 599]
    inp.x[zero_rows] = 0
    got = _run(inp, k, "zero tokens")
    assert np.all(got["m"][zero_rows] == 0.0)
    assert np.all(got["Z"][zero_rows] == float(M))  # M terms of exactly 1, exact in fp32
    _check_routing(inp, k, got, "zero tokens")
    _check_stats(inp, k, got, "zero tokens")


def test_train_is_reproducible_and_matches_routing():
    """Two calls give the same bits; the routing outputs equal those of more_route_lowrank."""
    from gpu_util import route_lowrank
    T, h, r, M, k = 2000, 128, 64, 20000, 8
    inp = make_inputs(T, h, r, M, seed=41)
    a = _run(inp, k, "repeat 1")
    b = _run(inp, k, "repeat 2")
    for n in ("idx", "gate", "topval", "counts", "m", "Z", "psum"):
        assert np.array_equal(a[n], b[n]), n
    idx, gate, topval, counts = route_lowrank(inp, k, histogram=True, tag="routing only")
    assert np.array_equal(a["idx"], idx) and np.array_equal(a["gate"], gate)
    assert np.array_equal(a["topval"], topval) and np.array_equal(a["counts"], counts)


def test_train_without_topval_and_histogram():
    T, h, r, M, k = 700, 64, 16, 2500, 8
    inp = make_inputs(T, h, r, M, seed=51)
    got = _run(inp, k, "no topval", topval=False, histogram=False)
    assert got["topval"] is None and got["counts"] is None
    _check_routing(inp, k, got, "no topval")
    _check_stats(inp, k, got, "no topval")


def test_train_empty_batch_zeroes_psum():
    torch = require_gpu()
    from paper_2609_36301_amd import router
    h, r, M, k = 64, 16, 300, 4
    announce("empty batch route_lowrank_train T=0 M=%d" % M)
    tr = router.LowrankTrainRouter(0, h, r, M, k)
    tr.out.psum.fill_(7.0)
    x = torch.zeros((0, h), dtype=torch.bfloat16, device="cuda")
    R1t = torch.zeros((r, h), dtype=torch.bfloat16, device="cuda")
    R2t = torch.zeros((M, r), dtype=torch.bfloat16, device="cuda")
    out = tr(x, R1t, R2t)
    torch.cuda.synchronize()
    assert torch.all(out.psum == 0).item()
    assert torch.all(out.counts == 0).item()


@pytest.mark.parametrize("name", ["tiny", "teaser_prefill", "decode", "mid", "fine_grained"])
def test_train_full_size_workloads(name):
    """The routing workloads at full size: m, Z and psum of every token and expert against the
    oracle; routing on a sample of rows."""
    inp = make_workload_inputs(name)
    T, h, r, M = inp.shape
    k = WORKLOADS[name].k
    got = _run(inp, k, name)
    rows = np.unique(np.concatenate([np.arange(0, T, max(1, T // 512)), [T - 1]]))
    _check_routing(inp, k, dict(got, counts=None), name, rows=rows)
    _check_stats(inp, k, got, name)
