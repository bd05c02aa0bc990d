"""GPU parity of the dispatch bookkeeping (Sort + Count) against the oracle: offsets and sorted
positions bit for bit (marked `gpu`).

Cases span one, two and three radix passes (keys below 2^8, 2^16 and 2^24), the one counting
pass (keys below 2^13), ids outside the expert range, one expert taking every entry, entry counts that are not a multiple of the
1024-entry block, no tokens, the bench workloads' sizes with a skewed expert choice, and the
output of a routing call.
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, require_gpu, to_dev

pytestmark = pytest.mark.gpu


def _run(idx, M, tag):
    torch = require_gpu()
    from paper_2609_36301_amd import router
    announce("%s dispatch_sort T=%d k=%d M=%d" % (tag, idx.shape[0], idx.shape[1], M))
    offsets, srt = router.dispatch_sort(to_dev(np.ascontiguousarray(idx, np.int32)), M)
    torch.cuda.synchronize()
    return offsets.cpu().numpy(), srt.cpu().numpy()


def _check(idx, M, tag):
    got_o, got_s = _run(idx, M, tag)
    want_o, want_s = oracle.dispatch_sort(idx, M)
    assert np.array_equal(got_o.astype(np.int64), want_o), tag
    assert np.array_equal(got_s.astype(np.int64), want_s), tag
    print("[dispatch] %s T=%d k=%d M=%d ok" % (tag, idx.shape[0], idx.shape[1], M), flush=True)


def _skewed(T, k, M, seed):
    """Expert ids with a Zipf-like skew (a few experts take many entries)."""
    rng = np.random.default_rng(seed)
    w = 1.0 / np.arange(1, M + 1) ** 0.8
    cdf = np.cumsum(w / w.sum())
    perm = rng.permutation(M).astype(np.int32)
    pick = np.minimum(np.searchsorted(cdf, rng.random((T, k))), M - 1)
    return perm[pick]


@pytest.mark.parametrize("T,k,M", [(256, 8, 200), (256, 8, 256), (1001, 3, 5000),
                                   (4096, 4, 70000),
                                   # one counting pass (more than 4096 entries, M + 1 <= 8192)
                                   (16384, 8, 4096), (3000, 7, 8191), (20000, 3, 1),
                                   (1100, 4, 300), (5000, 2, 8192)],
                         ids=lambda v: str(v))
def test_random_ids(T, k, M):
    rng = np.random.default_rng(T + M)
    _check(rng.integers(0, M, size=(T, k)).astype(np.int32), M, "random")


@pytest.mark.parametrize("T,k,M", [(3000, 4, 8192), (5000, 3, 16384), (1100, 8, 40000),
                                   (2000, 4, 524287), (2100, 4, 524288)],
                         ids=lambda v: str(v))
def test_wide_keys_with_invalid_ids_and_a_hot_expert(T, k, M):
    # keys of 14 to 20 bits (two and three radix passes), ids outside [0, M) and a hot expert
    rng = np.random.default_rng(T + k + M)
    idx = rng.integers(0, M, size=(T, k)).astype(np.int32)
    idx[::13, 0] = -1
    idx[::17, 1] = 2 ** 31 - 1
    idx[::3, 2] = M - 1
    _check(idx, M, "wide keys")


def test_sixteen_hot_experts_take_every_entry():
    rng = np.random.default_rng(8)
    idx = rng.integers(65520, 65536, size=(10000, 8)).astype(np.int32)
    _check(idx, 65536, "sixteen hot experts")


def test_ids_outside_the_range_go_last():
    rng = np.random.default_rng(3)
    idx = rng.integers(-5, 120, size=(777, 5)).astype(np.int32)
    idx[::7, 0] = 2 ** 31 - 1
    _check(idx, 100, "invalid ids")


def test_ids_outside_the_range_go_last_one_pass():
    rng = np.random.default_rng(4)
    idx = rng.integers(-3, 2000, size=(3000, 6)).astype(np.int32)
    idx[::5, 2] = 2 ** 31 - 1
    _check(idx, 1990, "outside, one pass")


def test_teaser_sized_skew_one_pass():
    _check(_skewed(16384, 8, 4096, seed=5), 4096, "skewed teaser")


def test_one_expert_takes_every_entry():
    idx = np.full((5000, 4), 17, np.int32)
    _check(idx, 1000, "one expert")


def test_no_tokens_writes_zero_offsets():
    o, s = _run(np.zeros((0, 8), np.int32), 300, "empty")
    assert s.size == 0 and np.array_equal(o, np.zeros(301, np.int32))


@pytest.mark.parametrize("T,k,M", [(32768, 8, 16384), (16384, 8, 65536), (128, 16, 262144)],
                         ids=["mid", "fine_grained", "decode"])
def test_workload_sizes_with_skew(T, k, M):
    _check(_skewed(T, k, M, seed=M), M, "skewed")


def test_routing_output():
    from gpu_util import route_lowrank
    from paper_2609_36301_amd.inputs import make_inputs
    inp = make_inputs(4096, 256, 32, 40000, seed=11, expert_bias_var=0.5)
    idx = route_lowrank(inp, 8, tag="dispatch input")[0]
    _check(idx, 40000, "routing output")
    a = _run(idx, 40000, "repeat")
    b = _run(idx, 40000, "repeat")
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
