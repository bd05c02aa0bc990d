"""GPU parity of the full-rank baseline router and of the expert histogram (marked `gpu`)."""
import numpy as np
import pytest

import oracle
from oracle import parity
from gpu_util import announce, require_gpu, to_dev
from paper_2609_36301_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits, make_inputs

pytestmark = pytest.mark.gpu


def _w_bf16(inp):
    """W = R1 R2 formed in fp64 on the host, rounded to bf16 ([h][M])."""
    W = bf16_bits_to_f32(inp.R1).astype(np.float64) @ bf16_bits_to_f32(inp.R2).astype(np.float64)
    return f32_to_bf16_bits(W.astype(np.float32))


def _fullrank(inp, Wb, k, bits, tag):
    torch = require_gpu()
    from paper_2609_36301_amd import router
    T, h = inp.x.shape
    M = Wb.shape[1]
    announce("%s route_fullrank T=%d h=%d M=%d k=%d logit_bits=%d" % (tag, T, h, M, k, bits))
    out = router.route_fullrank(to_dev(inp.x), to_dev(np.ascontiguousarray(Wb.T)), k,
                                topval=True, logit_bits=bits)
    torch.cuda.synchronize()
    return out.idx.cpu().numpy(), out.gate.cpu().numpy(), out.topval.cpu().numpy()


@pytest.mark.parametrize("shape", [(16384, 512, 32, 4096, 8), (333, 128, 16, 1000, 5),
                                   (500, 128, 16, 2048, 32), (64, 64, 16, 33, 32),
                                   (1, 32, 16, 7, 1)],
                         ids=lambda s: "T%d_h%d_M%d_k%d" % (s[0], s[1], s[3], s[4]))
def test_fullrank_fp32_logits_parity(shape):
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=5)
    Wb = _w_bf16(inp)
    idx, gate, topval = _fullrank(inp, Wb, k, 32, "fullrank")
    orc = oracle.route_fullrank(inp.x, Wb, k)
    picked = oracle.fullrank_logits_at(inp.x, Wb, np.arange(T), idx)
    rep = parity.compare(orc, idx, gate, k, M, picked, topval)
    print("[parity] fullrank %s %s" % (shape, rep), flush=True)
    assert rep.ok(), str(rep)


@pytest.mark.parametrize("bits", [32, 16])
def test_fullrank_exact_ties_keep_the_selection_order(bits):
    """Duplicated columns of W tie exactly: the row top-k must keep equal logits in expert-id
    order also when a later, larger logit shifts them down its register list."""
    T, h, r, M, k = 700, 256, 16, 3000, 8
    inp = make_inputs(T, h, r, M, seed=91)
    Wb = _w_bf16(inp)
    rng = np.random.default_rng(92)
    src = rng.choice(M, size=M // 10, replace=False)
    dst = rng.choice(np.setdiff1d(np.arange(M), src), size=src.size, replace=False)
    Wb[:, dst] = Wb[:, src]
    idx, gate, topval = _fullrank(inp, Wb, k, bits, "fullrank ties")
    parity.check_valid(idx, gate, M, topval)  # (logit descending, id ascending) order
    if bits == 32:
        orc = oracle.route_fullrank(inp.x, Wb, k)
        picked = oracle.fullrank_logits_at(inp.x, Wb, np.arange(T), idx)
        rep = parity.compare(orc, idx, gate, k, M, picked, topval)
        print("[parity] fullrank ties %s" % rep, flush=True)
        assert rep.ok(), str(rep)


@pytest.mark.parametrize("bits,M,k", [(32, 4096, 8), (16, 4096, 16), (32, 1000, 32),
                                      (16, 16384, 8)])
def test_fullrank_zero_tokens_tie_every_expert(bits, M, k):
    """All-zero tokens tie every expert at logit 0: more logits reach the short-row threshold than
    it holds, so those rows take the list path; the result is experts 0 .. k-1 with gates 1/k."""
    T, h, r = 300, 128, 16
    inp = make_inputs(T, h, r, M, seed=M + k)
    zero_rows = [0, 1, 63, 64, 299]
    inp.x[zero_rows] = 0
    Wb = _w_bf16(inp)
    idx, gate, topval = _fullrank(inp, Wb, k, bits, "fullrank zero tokens")
    parity.check_valid(idx, gate, M, topval)
    for t in zero_rows:
        assert np.array_equal(idx[t], np.arange(k, dtype=np.int32)), (t, idx[t])
        assert np.allclose(gate[t], 1.0 / k, atol=1e-7)
        assert np.all(topval[t] == 0.0)
    if bits == 32:
        orc = oracle.route_fullrank(inp.x, Wb, k)
        picked = oracle.fullrank_logits_at(inp.x, Wb, np.arange(T), idx)
        rep = parity.compare(orc, idx, gate, k, M, picked, topval)
        assert rep.ok(), str(rep)


@pytest.mark.parametrize("shape", [(2000, 512, 32, 4096, 8), (700, 256, 32, 1003, 16)],
                         ids=lambda s: "T%d_M%d_k%d" % (s[0], s[3], s[4]))
def test_fullrank_bf16_logits_valid(shape):
    """Rows of 4096 bf16 logits take the 16-byte path of the row top-k, rows of 1003 the
    one-logit path."""
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=6)
    Wb = _w_bf16(inp)
    idx, gate, topval = _fullrank(inp, Wb, k, 16, "fullrank-bf16")
    parity.check_valid(idx, gate, M, topval)
    orc = oracle.route_fullrank(inp.x, Wb, k)
    same = np.all(np.sort(orc.idx, 1) == np.sort(idx, 1), axis=1)
    # bf16 logits carry 8 significant bits: most sets still agree
    assert same.mean() > 0.8, same.mean()


@pytest.mark.parametrize("M,T,k,skew", [(64, 1000, 4, False), (16384, 32768, 8, False),
                                        (65536, 16384, 8, True), (262144, 128, 16, False),
                                        (100, 0, 3, False)])
def test_histogram(M, T, k, skew):
    torch = require_gpu()
    from paper_2609_36301_amd import router
    rng = np.random.default_rng(M + T)
    if skew:  # 40% of all selections on one expert
        idx = rng.integers(0, M, size=(T, k)).astype(np.int32)
        idx[:, 0] = np.where(rng.random(T) < 0.4 * k, 7, idx[:, 0])
    else:
        idx = rng.integers(0, M, size=(T, k)).astype(np.int32)
    announce("expert_histogram T=%d k=%d M=%d" % (T, k, M))
    counts = router.expert_histogram(to_dev(idx), M)
    torch.cuda.synchronize()
    c = counts.cpu().numpy()
    assert np.array_equal(c, oracle.histogram(idx, M).astype(np.int32))
