"""MoRE low-rank mixture-of-experts router for AMD Instinct MI355X (gfx950).

The compute lives in libmore.so (HIP kernels behind the C ABI declared in include/more.h).
This package holds the library, its build script (`python -m paper_2609_36301_amd.build`),
a ctypes binding with torch tensors (`router`), and the seeded input generator (`inputs`).

    from paper_2609_36301_amd import route_lowrank
    out = route_lowrank(x, R1t, R2t, k)      # out.idx [T][k] int32, out.gate [T][k] fp32
    tr = route_lowrank_train(x, R1t, R2t, k) # + tr.m, tr.Z [T], tr.psum [M] fp32
    gr = route_lowrank_backward(x, R1t, R2t, tr.idx, dtop, pbar, tr.m, tr.Z)  # gr.dx, gr.dR1t, gr.dR2t
"""
__all__ = ["route_lowrank", "route_lowrank_train", "route_fullrank", "route_fullrank_fused",
           "expert_histogram",
           "dispatch_sort", "LowrankRouter", "LowrankTrainRouter", "lowrank_workspace_size",
           "lowrank_train_workspace_size", "route_lowrank_backward", "LowrankBackward",
           "lowrank_backward_workspace_size", "Gradients", "lowrank_plan", "lowrank_route",
           "fullrank_workspace_size", "Routing", "TrainRouting"]


def __getattr__(name):
    if name in __all__:
        from . import router
        return getattr(router, name)
    raise AttributeError(name)
