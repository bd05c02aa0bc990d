"""The no-allocation entry point through the C ABI (marked `gpu`): two calls in a row, the
second on a smaller input (single-pass route, then resident route), then a call on the wide
route, each bitwise equal to more_route_lowrank with a torch-allocated workspace, and in
oracle parity."""
import ctypes

import numpy as np
import pytest

from oracle import parity
from paper_2609_36301_amd.inputs import make_inputs, transposed_factors

pytestmark = pytest.mark.gpu


def _run(lib, name, args, T, k, M, ws=None, wsb=0):
    import torch
    idx = torch.full((T, k), -7, dtype=torch.int32, device="cuda")
    gate = torch.full((T, k), -7.0, dtype=torch.float32, device="cuda")
    tv = torch.full((T, k), -7.0, dtype=torch.float32, device="cuda")
    cnt = torch.full((M,), 12345, dtype=torch.int32, device="cuda")
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    x_d, r1_d, r2_d, shape = args
    T_, h, r, M_, k_ = shape
    if name == "noalloc":
        st = lib.more_route_lowrank_noalloc(P(x_d), P(r1_d), P(r2_d), T_, h, r, M_, k_, P(idx),
                                            P(gate), P(tv), P(cnt), stream)
    else:
        st = lib.more_route_lowrank(P(x_d), P(r1_d), P(r2_d), T_, h, r, M_, k_, P(idx), P(gate),
                                    P(tv), P(cnt), None if ws is None else P(ws), wsb, stream)
    return st, (idx, gate, tv, cnt)


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    import torch
    from gpu_util import announce, require_gpu, to_dev
    from paper_2609_36301_amd import _lib
    require_gpu()
    lib = _lib.load()
    # the first call takes the single-pass route, the second (smaller) the resident route, on
    # scratch that still holds the first call's data
    for shape in ((4096, 512, 64, 40000, 8), (700, 256, 32, 9000, 16)):
        T, h, r, M, k = shape
        inp = make_inputs(T, h, r, M, seed=T + 11 * M)
        R1t, R2t = transposed_factors(inp)
        args = (to_dev(inp.x), to_dev(R1t), to_dev(R2t), shape)
        n = ctypes.c_size_t(0)
        assert lib.more_route_lowrank_workspace_size(T, h, r, M, k, ctypes.byref(n)) == _lib.OK
        assert 0 < n.value <= _lib.NOALLOC_SCRATCH_BYTES  # the scratch is really used
        announce("noalloc T=%d h=%d r=%d M=%d k=%d" % shape)
        st, got = _run(lib, "noalloc", args, T, k, M)
        assert st == _lib.OK, _lib.status_string(st)
        torch.cuda.synchronize()
        got = [t.cpu().numpy() for t in got]
        ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")
        announce("workspace entry point T=%d h=%d r=%d M=%d k=%d" % shape)
        st, want = _run(lib, "ws", args, T, k, M, ws, n.value)
        assert st == _lib.OK, _lib.status_string(st)
        torch.cuda.synchronize()
        want = [t.cpu().numpy() for t in want]
        for a, b in zip(got, want):
            assert np.array_equal(a, b)
        rep = parity.evaluate(inp.x, inp.R1, inp.R2, k, got[0], got[1], got[2])
        print("[parity] noalloc %s %s" % (shape, rep), flush=True)
        assert rep.ok(), str(rep)
        del args, ws


def test_noalloc_wide_route_matches_the_workspace_entry_point():
    # r = 128 with k = 20 takes the wide route; its z, split and list buffers come from the
    # same static scratch, which still holds the previous calls' data
    import torch
    from gpu_util import announce, require_gpu, to_dev
    from paper_2609_36301_amd import _lib, router
    require_gpu()
    lib = _lib.load()
    shape = (600, 256, 128, 3000, 20)
    T, h, r, M, k = shape
    assert router.lowrank_route(T, h, r, M, k) == "wide"
    inp = make_inputs(T, h, r, M, seed=17)
    R1t, R2t = transposed_factors(inp)
    args = (to_dev(inp.x), to_dev(R1t), to_dev(R2t), shape)
    n = ctypes.c_size_t(0)
    assert lib.more_route_lowrank_workspace_size(T, h, r, M, k, ctypes.byref(n)) == _lib.OK
    assert 0 < n.value <= _lib.NOALLOC_SCRATCH_BYTES
    announce("noalloc wide T=%d h=%d r=%d M=%d k=%d" % shape)
    st, got = _run(lib, "noalloc", args, T, k, M)
    assert st == _lib.OK, _lib.status_string(st)
    torch.cuda.synchronize()
    got = [t.cpu().numpy() for t in got]
    ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")
    st, want = _run(lib, "ws", args, T, k, M, ws, n.value)
    assert st == _lib.OK, _lib.status_string(st)
    torch.cuda.synchronize()
    want = [t.cpu().numpy() for t in want]
    for a, b in zip(got, want):
        assert np.array_equal(a, b)
    rep = parity.evaluate(inp.x, inp.R1, inp.R2, k, got[0], got[1], got[2])
    print("[parity] noalloc wide %s %s" % (shape, rep), flush=True)
    assert rep.ok(), str(rep)
