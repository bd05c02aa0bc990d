"""The C ABI on the host: symbols, validation and size queries (no GPU needed).

Every call here either fails validation or is a pure host query, so nothing is launched.
"""
import ctypes
import os
import re

import pytest

from paper_2609_36301_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "more.h")

FAKE = ctypes.c_void_p(0x10000)  # aligned, never dereferenced (validation fails first)
ODD = ctypes.c_void_p(0x10002)  # misaligned


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_36301_amd import build
        build.build(verbose=False)
    return _lib.load()


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:more_status|const char\*)\s+(more_\w+)\(", text, re.M)))


def test_header_declares_the_api():
    names = declared_symbols()
    for n in ("more_route_lowrank", "more_route_fullrank", "more_expert_histogram",
              "more_route_lowrank_workspace_size", "more_status_string"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), name
        assert name in _lib.SIGNATURES, "binding lacks " + name


def test_status_strings(lib):
    for s in range(5):
        assert lib.more_status_string(s)
    assert lib.more_status_string(99).startswith(b"MORE_ERR_UNKNOWN")
    assert b"gfx950" in lib.more_version()


def lowrank(lib, T=64, h=64, r=16, M=64, k=4, x=FAKE, R1t=FAKE, R2t=FAKE, idx=FAKE, gate=FAKE,
            topval=None, counts=None, ws=None, wsb=0, m_chunks=0):
    return lib.more_route_lowrank_ex(x, R1t, R2t, T, h, r, M, k, m_chunks, idx, gate, topval,
                                     counts, ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), _lib.ERR_INVALID_ARG),
    (dict(R1t=None), _lib.ERR_INVALID_ARG),
    (dict(R2t=None), _lib.ERR_INVALID_ARG),
    (dict(idx=None), _lib.ERR_INVALID_ARG),
    (dict(gate=None), _lib.ERR_INVALID_ARG),
    (dict(x=ODD), _lib.ERR_INVALID_ARG),
    (dict(R2t=ODD), _lib.ERR_INVALID_ARG),
    (dict(idx=ctypes.c_void_p(0x10001)), _lib.ERR_INVALID_ARG),
    (dict(T=-1), _lib.ERR_INVALID_ARG),
    (dict(h=0), _lib.ERR_INVALID_ARG),
    (dict(r=0), _lib.ERR_INVALID_ARG),
    (dict(M=0), _lib.ERR_INVALID_ARG),
    (dict(k=0), _lib.ERR_INVALID_ARG),
    (dict(k=65, M=64), _lib.ERR_INVALID_ARG),
    (dict(k=33, M=64), _lib.ERR_UNSUPPORTED),
    (dict(r=40), _lib.ERR_UNSUPPORTED),
    (dict(r=272), _lib.ERR_UNSUPPORTED),
    (dict(h=72), _lib.ERR_UNSUPPORTED),
    # the wide route's shapes pass validation and then need their workspace
    (dict(k=17, M=64), _lib.ERR_WORKSPACE),
    (dict(k=32, M=64), _lib.ERR_WORKSPACE),
    (dict(r=48), _lib.ERR_WORKSPACE),
    (dict(r=128), _lib.ERR_WORKSPACE),
    (dict(r=256), _lib.ERR_WORKSPACE),
    (dict(T=2**31), _lib.ERR_UNSUPPORTED),
    (dict(m_chunks=3), _lib.ERR_INVALID_ARG),
    (dict(m_chunks=2048), _lib.ERR_INVALID_ARG),
    (dict(m_chunks=-1), _lib.ERR_INVALID_ARG),
])
def test_lowrank_validation(lib, kw, status):
    assert lowrank(lib, **kw) == status


def test_lowrank_empty_batch_is_a_no_op(lib):
    assert lowrank(lib, T=0) == _lib.OK
    # an empty batch's token buffers may be NULL (torch gives empty tensors no storage)
    assert lowrank(lib, T=0, x=None, idx=None, gate=None) == _lib.OK
    assert lowrank(lib, T=0, R2t=None) == _lib.ERR_INVALID_ARG


def test_lowrank_workspace_checked_before_launch(lib):
    n = ctypes.c_size_t(0)
    assert lib.more_route_lowrank_workspace_size_ex(1000, 512, 32, 4096, 8, 8,
                                                    ctypes.byref(n)) == _lib.OK
    assert n.value > 0
    assert lowrank(lib, T=1000, h=512, r=32, M=4096, k=8, m_chunks=8) == _lib.ERR_WORKSPACE
    assert lowrank(lib, T=1000, h=512, r=32, M=4096, k=8, m_chunks=8, ws=FAKE,
                   wsb=n.value - 1) == _lib.ERR_WORKSPACE


def test_workspace_size_queries(lib):
    n = ctypes.c_size_t(123)
    assert lib.more_route_lowrank_workspace_size(0, 512, 32, 4096, 8, ctypes.byref(n)) == _lib.OK
    assert n.value == 0
    assert lib.more_route_lowrank_workspace_size(16, 512, 32, 4096, 8, None) == _lib.ERR_INVALID_ARG
    assert lib.more_route_lowrank_workspace_size(16, 512, 40, 4096, 8,
                                                 ctypes.byref(n)) == _lib.ERR_UNSUPPORTED
    # one big z buffer plus, for split plans, the chunk lists: grows with T
    a, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    lib.more_route_lowrank_workspace_size_ex(1024, 512, 32, 4096, 8, 8, ctypes.byref(a))
    lib.more_route_lowrank_workspace_size_ex(2048, 512, 32, 4096, 8, 8, ctypes.byref(b))
    assert b.value > a.value
    f = ctypes.c_size_t(0)
    assert lib.more_route_fullrank_workspace_size(100, 64, 1000, 4, 32, ctypes.byref(f)) == _lib.OK
    assert f.value >= 100 * 1000 * 4
    f16 = ctypes.c_size_t(0)
    assert lib.more_route_fullrank_workspace_size(100, 64, 1000, 4, 16, ctypes.byref(f16)) == 0
    assert f16.value < f.value
    assert lib.more_route_fullrank_workspace_size(100, 64, 1000, 4, 8,
                                                  ctypes.byref(f)) == _lib.ERR_INVALID_ARG


def test_plans_for_the_paper_shapes(lib):
    c = ctypes.c_int32(0)
    plans = {}
    for name, (T, h, r, M, k) in {"teaser": (16384, 512, 32, 4096, 8),
                                  "mid": (32768, 2048, 64, 16384, 8),
                                  "fine": (16384, 4096, 64, 65536, 8),
                                  "decode": (128, 4096, 64, 262144, 16)}.items():
        assert lib.more_route_lowrank_plan(T, h, r, M, k, ctypes.byref(c)) == _lib.OK
        plans[name] = c.value
    shapes = {"teaser": (16384, 32, 4096, 8), "mid": (32768, 64, 16384, 8),
              "fine": (16384, 64, 65536, 8), "decode": (128, 64, 262144, 16)}
    for name, C in plans.items():
        T, r, M, k = shapes[name]
        if r * M <= 1 << 18:  # fused route: 64 tokens per workgroup, the whole expert axis
            assert C == 0, name
            assert -(-T // 64) >= 256, name
            continue
        if T >= 4096 and M >= 32768:  # single-pass route
            assert C == 0, name
            continue
        tokens_per_block = 512  # 8 waves x 32 tokens x 2 token groups
        assert C & (C - 1) == 0, name
        assert r * M * 2 // C <= 2 << 20, name          # expert slice fits one L2
        assert C * -(-T // tokens_per_block) >= 256, name  # at least one workgroup per CU


def test_routes_for_the_paper_shapes(lib):
    from paper_2609_36301_amd import router
    want = {(16384, 512, 32, 4096, 8): "fused-local", (32768, 2048, 64, 16384, 8): "expert-resident",
            (16384, 4096, 64, 65536, 8): "single-pass", (128, 4096, 64, 262144, 16): "expert-resident",
            (4096, 256, 32, 32768, 8): "single-pass", (4095, 256, 32, 32768, 8): "expert-resident",
            (4096, 256, 32, 32767, 8): "expert-resident"}
    for shape, name in want.items():
        assert router.lowrank_route(*shape) == name, shape
    c = ctypes.c_int32(0)
    assert lib.more_route_lowrank_route(100, 64, 40, 1000, 4, ctypes.byref(c)) == _lib.ERR_UNSUPPORTED
    for r, k in ((48, 4), (128, 8), (256, 32), (16, 17), (64, 32)):
        assert lib.more_route_lowrank_route(100, 64, r, 1000, k, ctypes.byref(c)) == _lib.OK
        assert c.value == _lib.ROUTE_WIDE, (r, k)
        assert router.lowrank_route(100, 64, r, 1000, k) == "wide"
        mc = ctypes.c_int32(-1)
        assert lib.more_route_lowrank_plan(100, 64, r, 1000, k, ctypes.byref(mc)) == _lib.OK
        assert mc.value == 0
    assert lib.more_route_lowrank_route(100, 64, 32, 1000, 4, None) == _lib.ERR_INVALID_ARG


def test_wide_route_workspace_sizes(lib):
    # the wide route needs z, its three-piece split and (r not a multiple of 64) the stacked
    # expert rows: more bytes for more tokens, for more experts when stacked, and at least z
    n = ctypes.c_size_t(0)
    sizes = {}
    for T, h, r, M, k in ((1000, 256, 128, 3000, 8), (2000, 256, 128, 3000, 8),
                          (1000, 256, 80, 3000, 8), (1000, 256, 80, 6000, 8),
                          (1000, 256, 64, 3000, 20)):
        assert lib.more_route_lowrank_workspace_size(T, h, r, M, k, ctypes.byref(n)) == _lib.OK
        assert n.value >= T * r * 4 + T * 3 * r * 2
        sizes[(T, r, M, k)] = n.value
    assert sizes[(2000, 128, 3000, 8)] > sizes[(1000, 128, 3000, 8)]
    assert sizes[(1000, 80, 6000, 8)] - sizes[(1000, 80, 3000, 8)] >= 3000 * 3 * 80 * 2
    # one byte short of the size query: refused before any launch
    assert lowrank(lib, T=1000, h=256, r=128, M=3000, k=8, ws=FAKE,
                   wsb=sizes[(1000, 128, 3000, 8)] - 1) == _lib.ERR_WORKSPACE


def test_fullrank_validation(lib):
    def call(**kw):
        a = dict(x=FAKE, W=FAKE, T=10, h=64, M=100, k=4, bits=32, idx=FAKE, gate=FAKE, ws=None,
                 wsb=0)
        a.update(kw)
        return lib.more_route_fullrank(a["x"], a["W"], a["T"], a["h"], a["M"], a["k"], a["bits"],
                                       a["idx"], a["gate"], None, a["ws"], a["wsb"], None)
    assert call(x=None) == _lib.ERR_INVALID_ARG
    assert call(W=ODD) == _lib.ERR_INVALID_ARG
    assert call(k=101) == _lib.ERR_INVALID_ARG
    assert call(k=40) == _lib.ERR_UNSUPPORTED
    assert call(bits=8) == _lib.ERR_INVALID_ARG
    assert call() == _lib.ERR_WORKSPACE
    assert call(T=0) == _lib.OK


def test_histogram_validation(lib):
    assert lib.more_expert_histogram(FAKE, 10, 4, 100, None, None) == _lib.ERR_INVALID_ARG
    assert lib.more_expert_histogram(None, 10, 4, 100, FAKE, None) == _lib.ERR_INVALID_ARG
    assert lib.more_expert_histogram(FAKE, -1, 4, 100, FAKE, None) == _lib.ERR_INVALID_ARG
    assert lib.more_expert_histogram(FAKE, 10, 0, 100, FAKE, None) == _lib.ERR_INVALID_ARG
    assert lib.more_expert_histogram(FAKE, 10, 4, 0, FAKE, None) == _lib.ERR_INVALID_ARG
    assert lib.more_expert_histogram(ODD, 10, 4, 100, FAKE, None) == _lib.ERR_INVALID_ARG


def test_dispatch_sort_validation(lib):
    n = ctypes.c_size_t(0)
    assert lib.more_dispatch_sort_workspace_size(1000, 8, 5000, ctypes.byref(n)) == _lib.OK
    assert n.value >= 4 * 8000 * 4  # keys and positions, two buffers each
    assert lib.more_dispatch_sort_workspace_size(0, 8, 5000, ctypes.byref(n)) == _lib.OK
    assert n.value == 0
    assert lib.more_dispatch_sort_workspace_size(1 << 29, 8, 5000,
                                                 ctypes.byref(n)) == _lib.ERR_UNSUPPORTED
    assert lib.more_dispatch_sort_workspace_size(10, 0, 5000, ctypes.byref(n)) == _lib.ERR_INVALID_ARG
    assert lib.more_dispatch_sort_workspace_size(10, 4, 0, ctypes.byref(n)) == _lib.ERR_INVALID_ARG
    # checked on the host before anything is launched
    assert lib.more_dispatch_sort(FAKE, 10, 4, 100, None, FAKE, FAKE, 1 << 20,
                                  None) == _lib.ERR_INVALID_ARG
    assert lib.more_dispatch_sort(None, 10, 4, 100, FAKE, FAKE, FAKE, 1 << 20,
                                  None) == _lib.ERR_INVALID_ARG
    assert lib.more_dispatch_sort(FAKE, 10, 4, 100, FAKE, None, FAKE, 1 << 20,
                                  None) == _lib.ERR_INVALID_ARG
    assert lib.more_dispatch_sort(FAKE, -1, 4, 100, FAKE, FAKE, FAKE, 1 << 20,
                                  None) == _lib.ERR_INVALID_ARG
    assert lib.more_dispatch_sort(ODD, 10, 4, 100, FAKE, FAKE, FAKE, 1 << 20,
                                  None) == _lib.ERR_INVALID_ARG
    assert lib.more_dispatch_sort(FAKE, 10, 4, 100, FAKE, FAKE, None, 0,
                                  None) == _lib.ERR_WORKSPACE
    assert lib.more_dispatch_sort(FAKE, 10, 4, 100, FAKE, FAKE, FAKE, 16,
                                  None) == _lib.ERR_WORKSPACE


def train(lib, T=64, h=64, r=16, M=64, k=4, x=FAKE, idx=FAKE, gate=FAKE, m=FAKE, Z=FAKE,
          psum=FAKE, ws=FAKE, wsb=1 << 30):
    return lib.more_route_lowrank_train(x, FAKE, FAKE, T, h, r, M, k, idx, gate, None, None, m,
                                        Z, psum, ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), _lib.ERR_INVALID_ARG),
    (dict(idx=None), _lib.ERR_INVALID_ARG),
    (dict(m=None), _lib.ERR_INVALID_ARG),
    (dict(Z=None), _lib.ERR_INVALID_ARG),
    (dict(psum=None), _lib.ERR_INVALID_ARG),
    (dict(psum=ctypes.c_void_p(0x10002)), _lib.ERR_INVALID_ARG),
    (dict(ws=ctypes.c_void_p(0x10010)), _lib.ERR_INVALID_ARG),  # workspace: 256-byte aligned
    (dict(T=-1), _lib.ERR_INVALID_ARG),
    (dict(k=0), _lib.ERR_INVALID_ARG),
    (dict(k=17), _lib.ERR_UNSUPPORTED),
    (dict(r=48), _lib.ERR_UNSUPPORTED),
    (dict(ws=None, wsb=0), _lib.ERR_WORKSPACE),
    (dict(wsb=1000), _lib.ERR_WORKSPACE),
])
def test_train_validation(lib, kw, status):
    assert train(lib, **kw) == status


def test_train_workspace_size(lib):
    n, route = ctypes.c_size_t(7), ctypes.c_size_t(0)
    assert lib.more_route_lowrank_train_workspace_size(0, 512, 32, 4096, 8,
                                                       ctypes.byref(n)) == _lib.OK
    assert n.value == 0
    assert lib.more_route_lowrank_train_workspace_size(16, 512, 32, 4096, 8,
                                                       None) == _lib.ERR_INVALID_ARG
    for T, h, r, M, k in [(256, 512, 16, 256, 8), (16384, 512, 32, 4096, 8),
                          (32768, 2048, 64, 16384, 8), (16384, 4096, 64, 65536, 8),
                          (128, 4096, 64, 262144, 16)]:
        assert lib.more_route_lowrank_train_workspace_size(T, h, r, M, k,
                                                           ctypes.byref(n)) == _lib.OK
        assert lib.more_route_lowrank_workspace_size(T, h, r, M, k, ctypes.byref(route)) == 0
        # the route's workspace, then at least an internal top-k buffer, z' hi/lo, the per-chunk
        # normaliser partials and the psum partials
        assert n.value >= route.value + T * k * 4 + T * r * 4 + T * 4 + M * 4
    # workspace one byte short of the query is refused before any launch
    assert lib.more_route_lowrank_train_workspace_size(64, 64, 16, 64, 4, ctypes.byref(n)) == 0
    assert train(lib, wsb=n.value - 1) == _lib.ERR_WORKSPACE


def test_fullrank_fused_validation(lib):
    n = ctypes.c_size_t(0)
    # one token block of 100 tokens against 40000 experts: many expert splits, lists in workspace
    assert lib.more_route_fullrank_fused_workspace_size(100, 256, 40000, 8, ctypes.byref(n)) == 0
    assert n.value > 0
    assert lib.more_route_fullrank_fused_workspace_size(0, 256, 40000, 8, ctypes.byref(n)) == 0
    assert n.value == 0
    # the x rows of 32 tokens must fit a workgroup's LDS: h <= 2112
    assert lib.more_route_fullrank_fused_workspace_size(100, 2112, 4000, 8, ctypes.byref(n)) == 0
    assert lib.more_route_fullrank_fused_workspace_size(
        100, 2128, 4000, 8, ctypes.byref(n)) == _lib.ERR_UNSUPPORTED
    assert lib.more_route_fullrank_fused_workspace_size(
        100, 512, 4000, 33, ctypes.byref(n)) == _lib.ERR_UNSUPPORTED
    assert lib.more_route_fullrank_fused_workspace_size(100, 72, 4000, 8,
                                                        ctypes.byref(n)) == _lib.ERR_UNSUPPORTED
    call = lambda **kw: lib.more_route_fullrank_fused(
        kw.get("x", FAKE), kw.get("Wt", FAKE), kw.get("T", 100), kw.get("h", 256),
        kw.get("M", 40000), kw.get("k", 8), kw.get("idx", FAKE), kw.get("gate", FAKE), None,
        kw.get("ws", FAKE), kw.get("wsb", 1 << 30), None)
    assert call(x=None) == _lib.ERR_INVALID_ARG
    assert call(Wt=ODD) == _lib.ERR_INVALID_ARG
    assert call(k=0) == _lib.ERR_INVALID_ARG
    assert call(h=4096) == _lib.ERR_UNSUPPORTED
    assert call(ws=None, wsb=0) == _lib.ERR_WORKSPACE
    assert call(T=0, x=None, idx=None, gate=None) == _lib.OK


def backward(lib, T=64, h=64, r=16, M=64, k=4, x=FAKE, idx=FAKE, dtop=FAKE, pbar=FAKE, m=FAKE,
             Z=FAKE, dx=FAKE, dR1t=FAKE, dR2t=FAKE, ws=FAKE, wsb=1 << 30):
    return lib.more_route_lowrank_backward(x, FAKE, FAKE, T, h, r, M, k, idx, dtop, pbar, m, Z,
                                           dx, dR1t, dR2t, ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), _lib.ERR_INVALID_ARG),
    (dict(idx=None), _lib.ERR_INVALID_ARG),
    (dict(dtop=None), _lib.ERR_INVALID_ARG),
    (dict(dx=None), _lib.ERR_INVALID_ARG),
    (dict(dR1t=None), _lib.ERR_INVALID_ARG),
    (dict(dR2t=None), _lib.ERR_INVALID_ARG),
    (dict(m=None), _lib.ERR_INVALID_ARG),          # pbar given: the statistics are required
    (dict(Z=None), _lib.ERR_INVALID_ARG),
    (dict(dtop=ODD), _lib.ERR_INVALID_ARG),
    (dict(ws=ctypes.c_void_p(0x10010)), _lib.ERR_INVALID_ARG),
    (dict(T=-1), _lib.ERR_INVALID_ARG),
    (dict(k=0), _lib.ERR_INVALID_ARG),
    (dict(k=65), _lib.ERR_INVALID_ARG),            # k > M
    (dict(M=100, k=33), _lib.ERR_UNSUPPORTED),
    (dict(r=48), _lib.ERR_UNSUPPORTED),
    (dict(h=72), _lib.ERR_UNSUPPORTED),
    (dict(ws=None, wsb=0), _lib.ERR_WORKSPACE),
    (dict(wsb=1000), _lib.ERR_WORKSPACE),
])
def test_backward_validation(lib, kw, status):
    assert backward(lib, **kw) == status


def test_backward_workspace_size(lib):
    n, nb = ctypes.c_size_t(7), ctypes.c_size_t(0)
    assert lib.more_route_lowrank_backward_workspace_size(0, 512, 32, 4096, 8, 1,
                                                          ctypes.byref(n)) == _lib.OK
    assert n.value == 0
    assert lib.more_route_lowrank_backward_workspace_size(16, 512, 32, 4096, 8, 1,
                                                          None) == _lib.ERR_INVALID_ARG
    for T, h, r, M, k in [(256, 512, 16, 256, 8), (16384, 512, 32, 4096, 8),
                          (32768, 2048, 64, 16384, 8), (16384, 4096, 64, 65536, 8),
                          (128, 4096, 64, 262144, 16)]:
        assert lib.more_route_lowrank_backward_workspace_size(T, h, r, M, k, 1,
                                                              ctypes.byref(n)) == _lib.OK
        assert lib.more_route_lowrank_backward_workspace_size(T, h, r, M, k, 0,
                                                              ctypes.byref(nb)) == _lib.OK
        # z, z' hi/lo, dz hi/lo twice, the transposed R1 and the sorted selections at least;
        # the softmax sweeps add their partials of g and dz (and of dR2 with several token splits)
        base = T * r * 4 + T * r * 4 + 2 * T * r * 4 + h * r * 2 + T * k * 4
        assert nb.value >= base
        assert n.value >= nb.value + T * 4 + T * r * 4
    # without pbar the statistics may be NULL
    assert lib.more_route_lowrank_backward_workspace_size(64, 64, 16, 64, 4, 0,
                                                          ctypes.byref(nb)) == 0
    assert backward(lib, pbar=None, m=None, Z=None, wsb=nb.value - 1) == _lib.ERR_WORKSPACE
    assert lib.more_route_lowrank_backward_workspace_size(64, 64, 16, 64, 4, 1,
                                                          ctypes.byref(n)) == 0
    assert backward(lib, wsb=n.value - 1) == _lib.ERR_WORKSPACE


def test_binding_rejects_bad_tensors():
    import torch
    from paper_2609_36301_amd import router
    x = torch.zeros((4, 16), dtype=torch.bfloat16)
    with pytest.raises(ValueError):  # CPU tensors are refused before any library call
        router.route_lowrank(x, torch.zeros((16, 16), dtype=torch.bfloat16),
                             torch.zeros((8, 16), dtype=torch.bfloat16), 2)
    with pytest.raises(TypeError):
        router.route_lowrank(x.float(), x, x, 2)


def test_noalloc_rejects_shapes_beyond_its_scratch(lib):
    # checked on the host before anything is launched or looked up on a device
    T, h, r, M, k = 1 << 20, 64, 16, 65536, 8
    n = ctypes.c_size_t(0)
    assert lib.more_route_lowrank_workspace_size(T, h, r, M, k, ctypes.byref(n)) == _lib.OK
    assert n.value > _lib.NOALLOC_SCRATCH_BYTES
    assert lib.more_route_lowrank_noalloc(FAKE, FAKE, FAKE, T, h, r, M, k, FAKE, FAKE, None,
                                          None, None) == _lib.ERR_WORKSPACE
    assert lib.more_route_lowrank_noalloc(None, FAKE, FAKE, 10, h, r, M, k, FAKE, FAKE, None,
                                          None, None) == _lib.ERR_INVALID_ARG
    assert lib.more_route_lowrank_noalloc(FAKE, FAKE, FAKE, 0, h, r, M, k, FAKE, FAKE, None,
                                          None, None) == _lib.OK
