"""Helpers for GPU tests: move seeded inputs to the device and call the library's binding."""
from __future__ import annotations

import sys

import numpy as np


def announce(msg: str):
    """Name the case on stdout (flushed) before each GPU step."""
    print("[gpu] " + msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("a GPU test ran without a visible GPU")
    from paper_2609_36301_amd import _lib
    _lib.load()  # fails loudly if libmore.so was not built
    return torch


def to_dev(a: np.ndarray):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if t.dtype == torch.uint16:
        t = t.view(torch.bfloat16)
    return t.to("cuda")


def route_lowrank(inp, k, *, m_chunks=0, topval=True, histogram=False, tag=""):
    """Run the HIP low-rank router on RouterInputs; returns numpy (idx, gate, topval, counts)."""
    torch = require_gpu()
    from paper_2609_36301_amd import router
    from paper_2609_36301_amd.inputs import transposed_factors
    T, h, r, M = inp.shape
    R1t, R2t = transposed_factors(inp)
    announce("%s route_lowrank T=%d h=%d r=%d M=%d k=%d m_chunks=%d seed=%d"
             % (tag, T, h, r, M, k, m_chunks, inp.seed))
    x_d, r1_d, r2_d = to_dev(inp.x), to_dev(R1t), to_dev(R2t)
    out = router.route_lowrank(x_d, r1_d, r2_d, k, topval=topval, histogram=histogram,
                               m_chunks=m_chunks)
    torch.cuda.synchronize()
    res = (out.idx.cpu().numpy(), out.gate.cpu().numpy(),
           None if out.topval is None else out.topval.cpu().numpy(),
           None if out.counts is None else out.counts.cpu().numpy())
    del x_d, r1_d, r2_d, out
    return res
