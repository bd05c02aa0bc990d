"""GPU parity of the HIP low-rank router against the fp64 oracle (marked `gpu`).

Rules of comparison are in oracle/parity.py.  Sizes: every workload of the benchmark suite at
its full size with the oracle on all of its tokens, plus small ragged shapes that span several
tiles and a partial last tile on both the token and the expert axis.
"""
import numpy as np
import pytest

import oracle
import oracle_pins
from oracle import parity
from gpu_util import route_lowrank
from paper_2609_36301_amd.inputs import WORKLOADS, make_inputs, make_workload_inputs

pytestmark = pytest.mark.gpu


def _sample_rows(T, n, seed, extra=()):
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(T, size=min(n, T), replace=False).tolist())
    rows.update([0, T - 1])
    rows.update(int(e) for e in extra)
    return np.array(sorted(rows), dtype=np.int64)


def _check(inp, k, idx, gate, topval=None, rows=None, label=""):
    """Oracle parity (oracle/parity.py rules) on the given rows, all tokens when rows is None."""
    rep = parity.evaluate(inp.x, inp.R1, inp.R2, k, idx, gate, topval, rows=rows)
    print("[parity] %s %s" % (label, rep), flush=True)
    assert rep.ok(), "%s: %s mismatched rows %s band rows %s" % (
        label, rep, rep.mismatch_rows[:10], rep.band_rows[:10])
    return rep


@pytest.mark.parametrize("name", ["tiny", "teaser_prefill"])
def test_workload_all_tokens(name):
    w = WORKLOADS[name]
    inp = make_workload_inputs(name)
    idx, gate, topval, _ = route_lowrank(inp, w.k, tag=name)
    _check(inp, w.k, idx, gate, topval, label=name)


def test_workload_mid_all_tokens_with_duplicates_and_histogram():
    w = WORKLOADS["mid"]
    inp = make_workload_inputs("mid")
    idx, gate, topval, counts = route_lowrank(inp, w.k, histogram=True, tag="mid")
    # duplicated tokens give bit-identical outputs
    assert np.array_equal(idx[inp.dup_dst], idx[inp.dup_src])
    assert np.array_equal(gate[inp.dup_dst], gate[inp.dup_src])
    assert np.array_equal(counts, oracle.histogram(idx, w.M).astype(np.int32))
    _check(inp, w.k, idx, gate, topval, label="mid")


def test_workload_fine_grained_all_tokens_with_histogram():
    w = WORKLOADS["fine_grained"]
    inp = make_workload_inputs("fine_grained")
    idx, gate, topval, counts = route_lowrank(inp, w.k, histogram=True, tag="fine_grained")
    assert np.array_equal(counts, oracle.histogram(idx, w.M).astype(np.int32))
    assert counts.sum() == w.T * w.k
    _check(inp, w.k, idx, gate, topval, label="fine_grained")


def test_workload_decode_all_tokens():
    w = WORKLOADS["decode"]
    inp = make_workload_inputs("decode")
    idx, gate, topval, _ = route_lowrank(inp, w.k, tag="decode")
    _check(inp, w.k, idx, gate, topval, label="decode")


def test_workload_decode_finer_chunking_is_bitwise_identical():
    # full size: twice the library's expert chunks (512 instead of 256) give the same bits
    w = WORKLOADS["decode"]
    inp = make_workload_inputs("decode")
    base = route_lowrank(inp, w.k, tag="decode")
    finer = route_lowrank(inp, w.k, m_chunks=512, tag="decode chunks=512")
    for a, b in zip(base[:3], finer[:3]):
        assert np.array_equal(a, b)


# r = 128 and k > 16 in the register-tiled routes: their kernels spilled registers and the
# r = 128, k = 32 case faulted the GPU with a cause not shown, so those instantiations stay
# off.  Such shapes now take the wide route, whose own shapes are in test_gpu_wide.py; these
# cases stay skipped as the record of the fault.
_OUT_OF_LIMITS = pytest.mark.skip(reason="r = 128 / k > 16 register-tiled instantiation that "
                                  "faulted the GPU (cause not shown) stays off")

RAGGED = [
    # T, h, r, M, k
    (1, 16, 16, 1, 1),
    (1, 64, 32, 100, 5),
    pytest.param((33, 48, 16, 31, 31), marks=_OUT_OF_LIMITS),
    (33, 48, 16, 31, 16),
    (65, 128, 16, 16, 16),
    (100, 80, 32, 1000, 1),
    (129, 256, 64, 777, 2),
    pytest.param((300, 512, 128, 2049, 8), marks=_OUT_OF_LIMITS),
    (300, 512, 64, 2049, 8),
    pytest.param((200, 64, 128, 300, 32), marks=_OUT_OF_LIMITS),
    (200, 64, 64, 300, 16),
    (257, 96, 64, 4100, 16),
    (64, 32, 32, 64, 3),
]


@pytest.mark.parametrize("shape", RAGGED, ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_ragged_shapes(shape):
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=T + M)
    idx, gate, topval, counts = route_lowrank(inp, k, histogram=True, tag="ragged")
    _check(inp, k, idx, gate, topval, label="ragged %s" % (shape,))
    assert np.array_equal(counts, oracle.histogram(idx, M).astype(np.int32))


@pytest.mark.parametrize("chunks", [8, 16, 64])
def test_expert_chunking_is_bitwise_identical(chunks):
    inp = make_inputs(500, 256, 32, 5000, seed=9)
    base = route_lowrank(inp, 8, m_chunks=1, tag="chunks=1")
    other = route_lowrank(inp, 8, m_chunks=chunks, tag="chunks=%d" % chunks)
    for a, b in zip(base[:3], other[:3]):
        assert np.array_equal(a, b)
    _check(inp, 8, base[0], base[1], base[2], label="chunks")


@pytest.mark.parametrize("shape", [(300, 96, 32, 8000, 8), (200, 64, 16, 2000, 16),
                                   (129, 128, 64, 3000, 4)],
                         ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_fused_route_matches_resident_route_bitwise(shape):
    # m_chunks=0 picks the fused route kernel (fed by the z pass) on these expert sets;
    # m_chunks=1 forces the expert-resident route (screen, threshold, collect, finalize kernels).
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=T + 3 * M)
    fused = route_lowrank(inp, k, histogram=True, tag="fused")
    resident = route_lowrank(inp, k, histogram=True, m_chunks=1, tag="resident")
    for a, b in zip(fused, resident):
        assert np.array_equal(a, b)
    _check(inp, k, fused[0], fused[1], fused[2], label="fused %s" % (shape,))


@pytest.mark.parametrize("shape", [(16384, 512, 32, 4096, 8), (77, 64, 16, 1000, 5),
                                   (129, 128, 32, 33, 1), (500, 208, 64, 1000, 8),
                                   # h staged in LDS over several chunks, the last one partial
                                   (96, 1280, 16, 700, 6), (70, 1088, 64, 500, 8),
                                   (130, 2080, 32, 3000, 4)],
                         ids=lambda s: "T%d_h%d_r%d_M%d_k%d" % s)
def test_local_route_matches_resident_route(shape):
    # m_chunks=0 picks the one-launch local kernel here (z computed in the workgroup, h summed in
    # four quarters): the same selections as the resident route, logits equal to rounding.
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=T + 5 * M)
    local = route_lowrank(inp, k, histogram=True, tag="local")
    resident = route_lowrank(inp, k, histogram=True, m_chunks=1, tag="resident")
    same = np.all(local[0] == resident[0], axis=1)
    assert same.mean() >= 0.999, same.mean()
    scale = np.abs(resident[2][same]).max() + 1.0
    assert np.abs(local[2][same] - resident[2][same]).max() <= 1e-5 * scale
    assert np.abs(local[1][same] - resident[1][same]).max() <= 1e-5
    _check(inp, k, local[0], local[1], local[2], label="local %s" % (shape,))
    assert np.array_equal(local[3], oracle.histogram(local[0], M).astype(np.int32))


def test_repeat_runs_bitwise_identical():
    inp = make_inputs(1000, 512, 64, 3000, seed=12)
    a = route_lowrank(inp, 16, tag="run1")
    b = route_lowrank(inp, 16, tag="run2")
    for u, v in zip(a[:3], b[:3]):
        assert np.array_equal(u, v)


@pytest.mark.parametrize("shape", [(256, 512, 16, 256, 8), (2048, 2048, 64, 16384, 8)])
def test_exact_ties_resolve_to_lower_expert(shape):
    """Duplicated R2 columns give identical logits; the lower expert id must win."""
    T, h, r, M, k = shape
    inp = make_inputs(T, h, r, M, seed=77, dup_expert_frac=0.05)
    idx, gate, topval, _ = route_lowrank(inp, k, tag="ties")
    rows = np.arange(T)
    orc = oracle.route_lowrank(inp.x, inp.R1, inp.R2, k)
    rep = parity.compare_with(orc, inp.x, inp.R1, inp.R2, k, idx, gate, topval)
    print("[parity] ties %s %s" % (shape, rep), flush=True)
    assert rep.ok(), str(rep)
    # boundary exactly tied in the oracle and isolated from every other logit by 1e-3
    # relative: the tie itself must be resolved exactly as the oracle resolves it.
    R2f = oracle_pins.f64(inp.R2)
    logits = (oracle_pins.f64(inp.x[rows]) @ oracle_pins.f64(inp.R1)) @ R2f
    n_tie = 0
    for i, t in enumerate(rows):
        v = orc.kth[i]
        if orc.next[i] != v:
            continue
        others = logits[i][logits[i] != v]
        if np.min(np.abs(others - v)) < 1e-3 * abs(v):
            continue
        n_tie += 1
        assert set(idx[t].tolist()) == set(orc.idx[i].tolist()), (t, idx[t], orc.idx[i])
    print("[ties] isolated exact boundary ties checked: %d" % n_tie, flush=True)


def test_theorem1_construction_on_gpu():
    g, S, x, R1, R2 = oracle_pins.thm1_inputs(0)
    from paper_2609_36301_amd.inputs import RouterInputs
    inp = RouterInputs(x=x, R1=R1, R2=R2, dup_dst=np.zeros(0, np.int64),
                       dup_src=np.zeros(0, np.int64), seed=0)
    idx, gate, topval, _ = route_lowrank(inp, g["k"], tag="thm1")
    assert np.array_equal(idx[0], S)
    assert np.all(topval[0] == np.float32(g["selected_logit_bf16"]))
    assert np.all(gate[0] == np.float32(0.125))


def test_proposition1_top1_and_counts_on_gpu():
    """Sign-vector experts at r = 8 (embedded in rank 16 with zero rows; same logits)."""
    n = 65536
    g, x, R1, R2 = oracle_pins.prop1_inputs(n, seed=2)
    r = g["r"]
    R1p = np.zeros((R1.shape[0], 16), np.uint16)
    R1p[:, :r] = R1
    R2p = np.zeros((16, R2.shape[1]), np.uint16)
    R2p[:r] = R2
    from paper_2609_36301_amd.inputs import RouterInputs
    inp = RouterInputs(x=x, R1=R1p, R2=R2p, dup_dst=np.zeros(0, np.int64),
                       dup_src=np.zeros(0, np.int64), seed=2)
    idx1, gate1, _, _ = route_lowrank(inp, 1, tag="prop1 k=1")
    z = oracle_pins.f64(x)[:, :r]
    expect = ((z > 0).astype(np.int64) << np.arange(r)).sum(axis=1)
    assert np.array_equal(idx1[:, 0], expect)
    assert np.all(gate1 == 1.0)
    idx8, _, _, counts = route_lowrank(inp, g["k"], histogram=True, tag="prop1 k=8")
    assert counts.sum() == n * g["k"]
    assert np.abs(counts - g["mean_count"]).max() <= g["bound"]


def test_graph_capture_replays_match_eager():
    """Routing calls of three routes (fused local, expert-resident with 16 chunks, wide at
    r = 128, k = 20) captured in one HIP graph; every replay equals the eager result."""
    import torch
    from gpu_util import require_gpu, to_dev, announce
    from paper_2609_36301_amd import router
    from paper_2609_36301_amd.inputs import transposed_factors
    require_gpu()
    shapes = [(700, 512, 32, 4096, 8, 0), (300, 256, 64, 20000, 16, 16),
              (400, 128, 128, 3000, 20, 0)]
    routers, args, eager = [], [], []
    for T, h, r, M, k, chunks in shapes:
        inp = make_inputs(T, h, r, M, seed=T)
        R1t, R2t = transposed_factors(inp)
        a = (to_dev(inp.x), to_dev(R1t), to_dev(R2t))
        lr = router.LowrankRouter(T, h, r, M, k, histogram=True, topval=True, m_chunks=chunks)
        announce("graph eager T=%d M=%d chunks=%d" % (T, M, chunks))
        o = lr(*a)
        torch.cuda.synchronize()
        eager.append([t.clone() for t in (o.idx, o.gate, o.topval, o.counts)])
        routers.append(lr)
        args.append(a)
    announce("graph capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for lr, a in zip(routers, args):
            lr(*a)
    for rep in range(3):
        for lr in routers:  # scribble over outputs between replays
            lr.out.idx.fill_(-1)
            lr.out.gate.fill_(-1.0)
            lr.out.counts.fill_(12345)
        torch.cuda.synchronize()
        announce("graph replay %d" % rep)
        g.replay()
        torch.cuda.synchronize()
        for lr, ref in zip(routers, eager):
            o = lr.out
            for got, want in zip((o.idx, o.gate, o.topval, o.counts), ref):
                assert torch.equal(got, want), "replay %d differs from eager" % rep
        _ = torch.ones(1000, device="cuda").sum().item()  # eager work between replays


@pytest.mark.parametrize("chunks", [0, 8])
def test_uncertified_tokens_recomputed_exactly(chunks):
    """Zero-vector tokens have all logits equal to 0: every expert meets the candidate
    threshold, the candidate list overflows and the finalize kernel sweeps all experts
    exactly.  Expected result: experts 0..k-1 (ties go to the lower id), gates 1/k;
    neighbours stay correct."""
    T, h, r, M, k = 300, 256, 32, 2000, 8
    inp = make_inputs(T, h, r, M, seed=3)
    zero_rows = [5, 77, 200, 299]
    inp.x[zero_rows] = 0
    idx, gate, topval, _ = route_lowrank(inp, k, m_chunks=chunks, tag="degenerate")
    for t in zero_rows:
        assert np.array_equal(idx[t], np.arange(k, dtype=np.int32))
        assert np.allclose(gate[t], 1.0 / k, atol=1e-7)
        assert np.all(topval[t] == 0.0)
    _check(inp, k, idx, gate, topval, label="degenerate")


def test_plain_entry_point_through_the_c_abi():
    """more_route_lowrank and more_route_lowrank_ex(m_chunks=0) called directly through
    ctypes on torch buffers: identical bits, and oracle parity."""
    import ctypes
    import torch
    from gpu_util import announce, require_gpu, to_dev
    from paper_2609_36301_amd import _lib
    from paper_2609_36301_amd.inputs import transposed_factors
    require_gpu()
    lib = _lib.load()
    for (T, h, r, M, k) in ((700, 256, 32, 3000, 8), (300, 512, 64, 40000, 16)):
        inp = make_inputs(T, h, r, M, seed=T + M)
        R1t, R2t = transposed_factors(inp)
        x_d, r1_d, r2_d = to_dev(inp.x), to_dev(R1t), to_dev(R2t)
        n = ctypes.c_size_t(0)
        assert lib.more_route_lowrank_workspace_size(T, h, r, M, k, ctypes.byref(n)) == 0
        ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device="cuda")
        outs = []
        for name in ("more_route_lowrank", "more_route_lowrank_ex"):
            idx = torch.empty((T, k), dtype=torch.int32, device="cuda")
            gate = torch.empty((T, k), dtype=torch.float32, device="cuda")
            tv = torch.empty((T, k), dtype=torch.float32, device="cuda")
            cnt = torch.empty((M,), dtype=torch.int32, device="cuda")
            P = lambda t: ctypes.c_void_p(t.data_ptr())
            stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
            announce("c-abi %s T=%d h=%d r=%d M=%d k=%d" % (name, T, h, r, M, k))
            if name == "more_route_lowrank":
                st = lib.more_route_lowrank(P(x_d), P(r1_d), P(r2_d), T, h, r, M, k, P(idx),
                                            P(gate), P(tv), P(cnt), P(ws), n.value, stream)
            else:
                st = lib.more_route_lowrank_ex(P(x_d), P(r1_d), P(r2_d), T, h, r, M, k, 0,
                                               P(idx), P(gate), P(tv), P(cnt), P(ws), n.value,
                                               stream)
            assert st == _lib.OK, _lib.status_string(st)
            torch.cuda.synchronize()
            outs.append([t.cpu().numpy() for t in (idx, gate, tv, cnt)])
        for a, b in zip(*outs):
            assert np.array_equal(a, b)
        idx, gate, tv, cnt = outs[0]
        _check(inp, k, idx, gate, tv, label="c-abi %s" % ((T, h, r, M, k),))
        assert np.array_equal(cnt, oracle.histogram(idx, M).astype(np.int32))
