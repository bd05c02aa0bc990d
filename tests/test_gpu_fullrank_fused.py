"""GPU parity of the fused full-rank router (more_route_fullrank_fused) against the fp64 oracle of
the standard router on the same bf16 W (marked `gpu`), under the routing parity rules.

Shapes cover every token-block width (128, 64 and 32 tokens, chosen by h and k), h with and
without a partial 64-wide chunk (16, 32 and 48 left over, h below 64), ragged token and expert
counts, one and many expert splits (the merge kernel), k up to 32, and exact ties from duplicated
expert columns (the smaller id must win).
"""
import numpy as np
import pytest

import oracle
from oracle import parity
from gpu_util import announce, require_gpu, to_dev
from paper_2609_36301_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits, make_inputs

pytestmark = pytest.mark.gpu


def _w_bf16(inp, rng=None):
    """A router matrix W [h][M] in bf16: R1 R2 formed in fp64 (unit-variance logits)."""
    W = bf16_bits_to_f32(inp.R1).astype(np.float64) @ bf16_bits_to_f32(inp.R2).astype(np.float64)
    return f32_to_bf16_bits(W.astype(np.float32))


def _fused(x, Wb, k, tag):
    torch = require_gpu()
    from paper_2609_36301_amd import router
    T, h = x.shape
    M = Wb.shape[1]
    announce("%s route_fullrank_fused T=%d h=%d M=%d k=%d" % (tag, T, h, M, k))
    out = router.route_fullrank_fused(to_dev(x), to_dev(np.ascontiguousarray(Wb.T)), k,
                                      topval=True)
    torch.cuda.synchronize()
    return out.idx.cpu().numpy(), out.gate.cpu().numpy(), out.topval.cpu().numpy()


def _check(x, Wb, k, tag):
    T = x.shape[0]
    M = Wb.shape[1]
    idx, gate, topval = _fused(x, Wb, k, tag)
    orc = oracle.route_fullrank(x, Wb, k)
    picked = oracle.fullrank_logits_at(x, Wb, np.arange(T), idx)
    rep = parity.compare(orc, idx, gate, k, M, picked, topval)
    print("[parity] fullrank-fused %s %s" % (tag, rep), flush=True)
    assert rep.ok(), "%s: %s" % (tag, rep)
    return idx, topval


SHAPES = [
    (16384, 512, 4096, 8),   # the teaser workload: 128-token blocks, four expert splits
    (333, 128, 1000, 5),     # ragged tokens and experts
    (500, 128, 2048, 32),    # k = 32: 32-token blocks
    (64, 64, 33, 32),        # k = 32 with M = 33
    (1, 32, 7, 1),           # one token, h below one 64-wide chunk
    (300, 80, 500, 16),      # h % 64 = 16, 64-token blocks
    (130, 1040, 2000, 8),    # h % 64 = 16 at the 64-token block's largest h
    (257, 2096, 3000, 4),    # near the largest h (32-token blocks), h % 64 = 48
    (100, 256, 40000, 8),    # one token block, many expert splits
    (2000, 96, 4100, 2),     # h % 64 = 32
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "T%d_h%d_M%d_k%d" % s)
def test_fullrank_fused_parity(shape):
    T, h, M, k = shape
    inp = make_inputs(T, h, 16, M, seed=T + h + M)
    _check(inp.x, _w_bf16(inp), k, str(shape))


def test_fullrank_fused_exact_ties_resolve_to_lower_expert():
    """Duplicated columns of W give bitwise equal logits: of two tied experts the smaller id
    is selected first."""
    T, h, M, k = 700, 256, 3000, 8
    inp = make_inputs(T, h, 16, M, seed=91)
    Wb = _w_bf16(inp)
    rng = np.random.default_rng(92)
    src = rng.choice(M, size=M // 10, replace=False)
    dst = rng.choice(np.setdiff1d(np.arange(M), src), size=src.size, replace=False)
    Wb[:, dst] = Wb[:, src]
    idx, topval = _check(inp.x, Wb, k, "ties")
    pairs = dict(zip(dst.tolist(), src.tolist()))
    for t in range(T):
        sel = set(idx[t].tolist())
        for j, e in enumerate(idx[t]):
            e = int(e)
            if e in pairs:  # a copy of column pairs[e]: its twin ties it exactly
                twin = pairs[e]
                if twin < e:
                    assert twin in sel, (t, e, twin)
                    jt = list(idx[t]).index(twin)
                    assert jt < j and topval[t, jt] == topval[t, j], (t, e, twin)


def test_fullrank_fused_matches_unfused_selections():
    """The fused and the materialising router select the same experts wherever the k-th and
    (k+1)-th logits are not within rounding of each other."""
    torch = require_gpu()
    from paper_2609_36301_amd import router
    T, h, M, k = 4000, 512, 4096, 8
    inp = make_inputs(T, h, 32, M, seed=93)
    Wb = _w_bf16(inp)
    idx_f, _, tv_f = _fused(inp.x, Wb, k, "fused vs unfused")
    out = router.route_fullrank(to_dev(inp.x), to_dev(np.ascontiguousarray(Wb.T)), k, topval=True)
    torch.cuda.synchronize()
    same = np.all(idx_f == out.idx.cpu().numpy(), axis=1)
    assert same.mean() > 0.999, same.mean()
    assert np.allclose(tv_f[same], out.topval.cpu().numpy()[same], rtol=1e-5, atol=1e-6)
