"""GPU parity of the training backward pass (more_route_lowrank_backward) against the oracle,
element by element, within the tolerance derived below (marked `gpu`).

Tolerance.  m and Z are inputs (the oracle's statistics rounded to fp32, given to both sides),
so P_te = exp(l_te - m_t) / Z_t differs between the two only through the recomputed logit.
With A_t = max_e |l_te|, S_t = max_e sum_i |z_ti u_ei| the exponent is within
    d_t = 1e-4 (1 + A_t) + 2^-18 S_t + (2r + 1) 2^-24 (A_t + S_t) + 2^-21 (|m_t| + |ln Z_t| + 1)
(the logit contract of z, the hi/lo rounding of z', the fp32 accumulation, and the fp32 bias
-(m log2 e + log2 Z)), so P is within D_t = expm1(d_t) + 2^-22 relative.  Then, with
G_t = sum_e |pbar_e| P_te and n = M + k + 1100 (terms and partials of an fp32 sum):
    |dg_t|  <= 1.01 (D_t + 2^-24 n) G_t
    |dy_te| <= E_te = P_te (|pbar_e - g_t| (D_t + 2^-8) + 1.02 |dg_t|)    (bf16 rounding 2^-9)
    |ddz_tj| <= tz_tj = sum_e E_te |u_je| + 1.1 2^-24 n (sum_e |y_te| |u_je|)
    |ddx_tc| <= sum_j tz_tj |R1_cj| + (2^-17 + 2^-24 (2r + 2)) sum_j |dz_tj| |R1_cj|
    |ddR1_cj| <= sum_t tz_tj |x_tc| + (2^-17 + 2^-24 (T + 1100)) sum_t |dz_tj| |x_tc|
    |ddR2_je| <= sum_t (E_te (1 + 2^-8) + 2^-8 |yd_te|) |z_tj| + sum_t |y_te| ez_tj
                 + 1.1 2^-24 (T + 1100) sum_t |y_te| |z_tj|
where yd is the dense part P (pbar - g), y = yd + the dtop scatter, dz_tj = sum_e y_te u_je,
ez_tj = (h + 64) 2^-24 sum_c |x_tc R1_cj| the fp32 error of z, and 2^-17 the hi/lo rounding of
dz.  A dropped term, a wrong sign or a transposed operand moves the results by far more.
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, require_gpu, to_dev
from paper_2609_36301_amd.inputs import (WORKLOADS, bf16_bits_to_f32, make_inputs,
                                         make_workload_inputs, transposed_factors)

pytestmark = pytest.mark.gpu


def f64(bits):
    return bf16_bits_to_f32(bits).astype(np.float64)


def _grad_inputs(inp, k, seed, balance=True, selection="oracle"):
    """idx (the oracle's routing, or a seeded synthetic selection of distinct experts), dtop,
    pbar = (M / T) f with f the selection frequency plus noise, and the oracle's m, Z in fp32."""
    T, h, r, M = inp.shape
    rng = np.random.default_rng(seed)
    if selection == "oracle":
        idx = oracle.route_lowrank(inp.x, inp.R1, inp.R2, k).idx.astype(np.int32)
    else:
        a = rng.integers(0, M, size=(T, 1))
        stride = rng.integers(1, max(2, M // k), size=(T, 1))
        idx = ((a + np.arange(k)[None, :] * stride) % M).astype(np.int32)
    dtop = rng.standard_normal((T, k)).astype(np.float32)
    pbar = m = Z = None
    if balance:
        f = np.bincount(idx[(idx >= 0) & (idx < M)], minlength=M) / max(1, T * k)
        pbar = ((M / max(T, 1)) * f + 0.3 * rng.random(M)).astype(np.float32)
        m64, Z64, _ = oracle.route_stats(inp.x, inp.R1, inp.R2)
        m, Z = m64.astype(np.float32), Z64.astype(np.float32)
    return idx, dtop, pbar, m, Z


def _run(inp, idx, dtop, pbar, m, Z, tag):
    torch = require_gpu()
    from paper_2609_36301_amd import router
    T, h, r, M = inp.shape
    k = idx.shape[1]
    R1t, R2t = transposed_factors(inp)
    announce("%s route_lowrank_backward T=%d h=%d r=%d M=%d k=%d seed=%d balance=%d"
             % (tag, T, h, r, M, k, inp.seed, pbar is not None))
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    out = router.route_lowrank_backward(to_dev(inp.x), to_dev(R1t), to_dev(R2t), dev(idx),
                                        dev(dtop), dev(pbar), dev(m), dev(Z))
    torch.cuda.synchronize()
    res = {n: getattr(out, n).cpu().numpy().astype(np.float64) for n in ("dx", "dR1t", "dR2t")}
    del out
    return res


def _tolerances(inp, idx, dtop, pbar, m, Z, g, dz, rows=None):
    """Per-element bounds of dx (rows `rows`, all by default), dR1 [h][r] and dR2 [r][M] from
    fp64 quantities in blocks of 256 tokens (dR1 and dR2 only when rows is None)."""
    T, h, r, M = inp.shape
    k = idx.shape[1]
    xf, R1, R2 = f64(inp.x), f64(inp.R1), f64(inp.R2)
    aR2, aR1 = np.abs(R2), np.abs(R1)
    rows = np.arange(T) if rows is None else np.asarray(rows)
    full = rows.size == T
    n = M + k + 1100
    tz = np.zeros((rows.size, r))
    tR2 = np.zeros((r, M))
    tR1 = np.zeros((h, r))
    for b0 in range(0, rows.size, 256):
        rr = rows[b0:b0 + 256]
        z = xf[rr] @ R1
        lg = z @ R2
        yd = np.zeros_like(lg)
        E = np.zeros_like(lg)
        if pbar is not None:
            A = np.abs(lg).max(axis=1)
            S = (np.abs(z) @ aR2).max(axis=1)
            mm, ZZ = m[rr].astype(np.float64), Z[rr].astype(np.float64)
            d = (1e-4 * (1 + A) + 2.0 ** -18 * S + (2 * r + 1) * 2.0 ** -24 * (A + S)
                 + 2.0 ** -21 * (np.abs(mm) + np.abs(np.log(ZZ)) + 1))
            D = np.expm1(d) + 2.0 ** -22
            P = np.exp(lg - mm[:, None]) / ZZ[:, None]
            pb = pbar.astype(np.float64)
            G = P @ np.abs(pb)
            dg = 1.01 * (D + 2.0 ** -24 * n) * G
            dev_ = pb[None, :] - g[rr][:, None]
            yd = P * dev_
            E = P * (np.abs(dev_) * (D + 2.0 ** -8)[:, None] + 1.02 * dg[:, None])
        y = yd.copy()
        for q in range(k):
            e = idx[rr, q]
            ok = (e >= 0) & (e < M)
            np.add.at(y, (np.nonzero(ok)[0], e[ok]), dtop[rr, q].astype(np.float64)[ok])
        tz[b0:b0 + 256] = E @ aR2.T + 1.1 * 2.0 ** -24 * n * (np.abs(y) @ aR2.T)
        if full:
            az = np.abs(z)
            ez = (h + 64) * 2.0 ** -24 * (np.abs(xf[rr]) @ aR1)
            tR2 += (az.T @ (E * (1 + 2.0 ** -8) + 2.0 ** -8 * np.abs(yd))
                    + ez.T @ np.abs(y) + 1.1 * 2.0 ** -24 * (T + 1100) * (az.T @ np.abs(y)))
            tR1 += (np.abs(xf[rr]).T @ tz[b0:b0 + 256]
                    + (2.0 ** -17 + 2.0 ** -24 * (T + 1100)) * (np.abs(xf[rr]).T @ np.abs(dz[rr])))
    tx = tz @ aR1.T + (2.0 ** -17 + 2.0 ** -24 * (2 * r + 2)) * (np.abs(dz[rows]) @ aR1.T)
    return tx, (tR1 if full else None), (tR2 if full else None)


def _compare(name, got, want, tol, tag):
    err = np.abs(got - want)
    bad = np.argwhere(err > tol + 1e-30)
    assert np.all(np.isfinite(got)), (tag, name, "non-finite")
    assert bad.size == 0, (tag, name, bad[:5].tolist(), err[tuple(bad[:5].T)], tol[tuple(bad[:5].T)])
    scale = np.abs(want).max() + 1e-30
    print("[backward] %s %s: max err %.3g (%.3g of max |grad|), max err/tol %.3g"
          % (tag, name, err.max(), err.max() / scale, (err / (tol + 1e-30)).max()), flush=True)


def _check_full(inp, idx, dtop, pbar, m, Z, got, tag):
    T, h, r, M = inp.shape
    f = lambda a: None if a is None else a.astype(np.float64)
    ref = oracle.route_backward(inp.x, inp.R1, inp.R2, idx, f(dtop), f(pbar), f(m), f(Z))
    tx, tR1, tR2 = _tolerances(inp, idx, dtop, pbar, m, Z, ref.g, ref.dz)
    _compare("dx", got["dx"], ref.dx, tx, tag)
    _compare("dR1", got["dR1t"].T, ref.dR1, tR1, tag)
    _compare("dR2", got["dR2t"].T, ref.dR2, tR2, tag)


SHAPES = [
    (256, 512, 16, 256, 8),      # tiny workload shape
    (300, 64, 16, 33, 2),        # ragged tokens, one full expert tile plus one expert
    (77, 64, 32, 5, 2),          # fewer experts than a tile
    (100, 32, 16, 1, 1),         # one expert: P = 1, the dense term vanishes
    (1000, 256, 32, 5000, 16),   # k = 16
    (513, 64, 64, 1100, 3),      # r = 64, ragged both ways
    (128, 256, 64, 9000, 16),    # decode-like: two token slots per workgroup
    (130, 128, 64, 2100, 8),     # one token past a slot boundary
    (2000, 128, 64, 20000, 8),   # many expert splits
    (300, 64, 32, 500, 32),      # k = 32 (the backward's limit)
    (20, 64, 32, 3000, 4),       # one token tile: dR2 written in place by the expert sweep
    (32, 128, 64, 40000, 8),     # the same with many expert blocks
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_backward_matches_oracle(shape):
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=600 + T % 97)
    ins = _grad_inputs(inp, k, seed=T)
    got = _run(inp, *ins, tag=str(shape))
    _check_full(inp, *ins, got, str(shape))


@pytest.mark.parametrize("shape", [(256, 512, 16, 256, 8), (513, 64, 64, 1100, 3)],
                         ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_backward_without_balancing_term(shape):
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=610)
    ins = _grad_inputs(inp, k, seed=3, balance=False)
    got = _run(inp, *ins, tag="nobal " + str(shape))
    _check_full(inp, *ins, got, "nobal " + str(shape))


def test_backward_invalid_and_repeated_ids():
    """ids outside [0, M) add nothing; an expert selected twice by a token gets both terms."""
    T, h, r, M, k = 200, 64, 32, 300, 4
    inp = make_inputs(T, h, r, M, seed=611)
    idx, dtop, pbar, m, Z = _grad_inputs(inp, k, seed=5)
    idx[::7, 1] = -1
    idx[3::11, 2] = M
    idx[5::13, 3] = idx[5::13, 0]
    got = _run(inp, idx, dtop, pbar, m, Z, tag="ids")
    _check_full(inp, idx, dtop, pbar, m, Z, got, "ids")


def test_backward_is_reproducible():
    T, h, r, M, k = 700, 128, 64, 3000, 8
    inp = make_inputs(T, h, r, M, seed=612)
    ins = _grad_inputs(inp, k, seed=6)
    a = _run(inp, *ins, tag="rep1")
    b = _run(inp, *ins, tag="rep2")
    for n in ("dx", "dR1t", "dR2t"):
        assert np.array_equal(a[n], b[n]), n


def test_backward_empty_batch():
    torch = require_gpu()
    from paper_2609_36301_amd import router
    T, h, r, M, k = 0, 64, 16, 40, 2
    inp = make_inputs(T, h, r, M, seed=613)
    R1t, R2t = transposed_factors(inp)
    announce("empty route_lowrank_backward")
    g = router.LowrankBackward(T, h, r, M, k, balance=True)
    g.out.dR1t.fill_(7.0)
    g.out.dR2t.fill_(7.0)
    e = lambda *s, dt=torch.float32: torch.zeros(s, dtype=dt, device="cuda")
    out = g(to_dev(inp.x), to_dev(R1t), to_dev(R2t), e(0, k, dt=torch.int32), e(0, k), e(M),
            e(0), e(0))
    torch.cuda.synchronize()
    assert not out.dR1t.any().item() and not out.dR2t.any().item()


@pytest.mark.parametrize("wl", ["teaser_prefill", "decode"])
def test_backward_full_workload(wl):
    """Every output element at the full workload size (synthetic distinct selections)."""
    inp = make_workload_inputs(wl)
    T, h, r, M = inp.shape
    k = WORKLOADS[wl].k
    ins = _grad_inputs(inp, k, seed=7, selection="synthetic")
    got = _run(inp, *ins, tag=wl)
    _check_full(inp, *ins, got, wl)


def _dr2_tolerance_cols(inp, cols, idx, dtop, pbar, m, Z, g):
    """The dR2 bound of the module docstring for the expert columns `cols` over all tokens, with
    A_t and S_t both replaced by their upper bound sum_i |z_ti| max_e |u_ie| (no T x M work)."""
    T, h, r, M = inp.shape
    k = idx.shape[1]
    xf, R1, R2 = f64(inp.x), f64(inp.R1), f64(inp.R2)
    tol = np.zeros((r, cols.size))
    colpos = {int(e): c for c, e in enumerate(cols)}
    umax = np.abs(R2).max(axis=1)
    for t0 in range(0, T, 2048):
        z = xf[t0:t0 + 2048] @ R1
        az = np.abs(z)
        Sb = az @ umax
        mm, ZZ = m[t0:t0 + 2048].astype(np.float64), Z[t0:t0 + 2048].astype(np.float64)
        d = (1e-4 * (1 + Sb) + 2.0 ** -18 * Sb + (2 * r + 1) * 2.0 ** -24 * 2 * Sb
             + 2.0 ** -21 * (np.abs(mm) + np.abs(np.log(ZZ)) + 1))
        D = np.expm1(d) + 2.0 ** -22
        lg = z @ R2[:, cols]
        P = np.exp(lg - mm[:, None]) / ZZ[:, None]
        dev_ = pbar.astype(np.float64)[cols][None, :] - g[t0:t0 + 2048][:, None]
        # |dg_t| needs G_t = sum_e |pbar_e| P_te over all experts; sum_e P_te = 1 bounds it
        G = np.abs(pbar).max() * np.ones_like(Sb)
        dg = 1.01 * (D + 2.0 ** -24 * (M + k + 1100)) * G
        yd = P * dev_
        E = P * (np.abs(dev_) * (D + 2.0 ** -8)[:, None] + 1.02 * dg[:, None])
        y = yd.copy()
        for q in range(k):
            e = idx[t0:t0 + 2048, q]
            for row in np.nonzero(np.isin(e, cols))[0]:
                y[row, colpos[int(e[row])]] += float(dtop[t0 + row, q])
        ez = (h + 64) * 2.0 ** -24 * (np.abs(xf[t0:t0 + 2048]) @ np.abs(R1))
        tol += (az.T @ (E * (1 + 2.0 ** -8) + 2.0 ** -8 * np.abs(yd)) + ez.T @ np.abs(y)
                + 1.1 * 2.0 ** -24 * (T + 1100) * (az.T @ np.abs(y)))
    return tol


@pytest.mark.parametrize("wl", ["mid", "fine_grained"])
def test_backward_full_workload_sampled(wl):
    """The oracle on the whole batch; dx on 64 sampled tokens and dR2 on 64 sampled experts
    (first, last and the most selected among them) element by element, and the trace identity
    <dx, x> = <dR1, R1> = <dR2, R2> over the whole batch, bounded by
    2^-6 sum_t A_t (2 max |pbar| + sum_j |dtop_tj|)."""
    inp = make_workload_inputs(wl)
    T, h, r, M = inp.shape
    k = WORKLOADS[wl].k
    idx, dtop, pbar, m, Z = _grad_inputs(inp, k, seed=8, selection="synthetic")
    got = _run(inp, idx, dtop, pbar, m, Z, tag=wl)
    f = lambda a: a.astype(np.float64)
    ref = oracle.route_backward(inp.x, inp.R1, inp.R2, idx, f(dtop), f(pbar), f(m), f(Z))
    rng = np.random.default_rng(9)
    rows = np.unique(np.concatenate([[0, T - 1], rng.integers(0, T, 62)]))
    tx, _, _ = _tolerances(inp, idx, dtop, pbar, m, Z, ref.g, ref.dz, rows=rows)
    _compare("dx (sampled rows)", got["dx"][rows], ref.dx[rows], tx, wl)
    hot = int(np.bincount(idx.ravel(), minlength=M).argmax())
    cols = np.unique(np.concatenate([[0, M - 1, hot], rng.integers(0, M, 61)]))
    t2 = _dr2_tolerance_cols(inp, cols, idx, dtop, pbar, m, Z, ref.g)
    _compare("dR2 (sampled experts)", got["dR2t"][cols].T, ref.dR2[:, cols], t2, wl)
    xf, R1, R2 = f64(inp.x), f64(inp.R1), f64(inp.R2)
    tx_ = np.sum(got["dx"] * xf)
    t1 = np.sum(got["dR1t"].T * R1)
    t2s = np.sum(got["dR2t"].T * R2)
    z = xf @ R1
    A = np.abs(z) @ np.abs(R2).max(axis=1)
    bound = 2.0 ** -6 * np.sum(A * (2 * np.abs(pbar).max() + np.abs(dtop).sum(axis=1)))
    print("[backward] %s trace identity: %.6g %.6g %.6g (bound %.3g)" % (wl, tx_, t1, t2s, bound),
          flush=True)
    assert abs(tx_ - t1) <= bound and abs(tx_ - t2s) <= bound


def test_backward_graph_replays_match_eager():
    """Two backward calls (with and without the balancing term) captured in one HIP graph; every
    replay, with the outputs scribbled over and eager work in between, equals the eager result."""
    torch = require_gpu()
    from paper_2609_36301_amd import router
    cases = []
    for T, h, r, M, k, bal in [(700, 256, 64, 5000, 8, True), (300, 128, 32, 3000, 4, False)]:
        inp = make_inputs(T, h, r, M, seed=T + 1)
        idx, dtop, pbar, m, Z = _grad_inputs(inp, k, seed=T, balance=bal)
        R1t, R2t = transposed_factors(inp)
        dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
        args = (to_dev(inp.x), to_dev(R1t), to_dev(R2t), dev(idx), dev(dtop), dev(pbar), dev(m),
                dev(Z))
        b = router.LowrankBackward(T, h, r, M, k, balance=bal)
        announce("backward graph eager T=%d M=%d balance=%d" % (T, M, bal))
        o = b(*args)
        torch.cuda.synchronize()
        cases.append((b, args, [t.clone() for t in (o.dx, o.dR1t, o.dR2t)]))
    announce("backward graph capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for b, args, _ in cases:
            b(*args)
    for rep in range(3):
        for b, _, _ in cases:
            for t in (b.out.dx, b.out.dR1t, b.out.dR2t):
                t.fill_(-7.0)
        torch.cuda.synchronize()
        announce("backward graph replay %d" % rep)
        g.replay()
        torch.cuda.synchronize()
        for b, _, ref in cases:
            for got, want in zip((b.out.dx, b.out.dR1t, b.out.dR2t), ref):
                assert torch.equal(got, want), "replay %d differs from eager" % rep
        _ = torch.ones(1000, device="cuda").sum().item()  # eager work between replays
