// C ABI of the router library: argument validation, planning and launch.
// Every check runs on the host before anything is enqueued, so an error status means the
// stream was not touched.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "more.h"
#include "lowrank.h"
#include "backward.h"
#include "wide.h"

namespace {

constexpr int64_t kMaxT = 0x7FFFFFFF;
constexpr int32_t kMaxM = 1 << 30;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool rank_supported(int32_t r) { return r == 16 || r == 32 || r == 64; }

more_status check_common(int64_t T, int32_t h, int32_t M, int32_t k) {
    if (T < 0 || h <= 0 || M <= 0 || k < 1 || k > M) return MORE_ERR_INVALID_ARG;
    if (T > kMaxT || M > kMaxM || h % 16 != 0 || k > MORE_K_MAX) return MORE_ERR_UNSUPPORTED;
    return MORE_OK;
}

// Inference calls take any r that is a multiple of 16 up to 256 and k <= 32 (the shapes outside
// the register-tiled routes go to the wide route); the training forward keeps those routes'
// limits, r in {16, 32, 64} and k <= 16.
more_status check_lowrank(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                          int32_t m_chunks, bool training = false) {
    if (r <= 0) return MORE_ERR_INVALID_ARG;
    more_status s = check_common(T, h, M, k);
    if (s != MORE_OK) return s;
    if (r % 16 != 0 || r > more::kWideMaxRank || k > MORE_LOWRANK_K_MAX) return MORE_ERR_UNSUPPORTED;
    if (training && (!rank_supported(r) || k > MORE_LOWRANK_TRAIN_K_MAX))
        return MORE_ERR_UNSUPPORTED;
    if (m_chunks < 0 || (m_chunks > 1 && (m_chunks % 8 != 0 || m_chunks > 1024)))
        return MORE_ERR_INVALID_ARG;
    return MORE_OK;
}

more_status from_hip(hipError_t e) { return e == hipSuccess ? MORE_OK : MORE_ERR_HIP; }

}  // namespace

extern "C" {

const char* more_status_string(more_status s) {
    switch (s) {
        case MORE_OK: return "MORE_OK";
        case MORE_ERR_INVALID_ARG: return "MORE_ERR_INVALID_ARG: invalid argument";
        case MORE_ERR_UNSUPPORTED: return "MORE_ERR_UNSUPPORTED: shape outside supported limits";
        case MORE_ERR_WORKSPACE: return "MORE_ERR_WORKSPACE: workspace missing or too small";
        case MORE_ERR_HIP: return "MORE_ERR_HIP: HIP runtime or hipBLASLt error";
    }
    return "MORE_ERR_UNKNOWN: unknown status";
}

const char* more_version(void) { return "0.1.0 gfx950"; }

more_status more_route_lowrank_workspace_size_ex(int64_t T, int32_t h, int32_t r, int32_t M,
                                                 int32_t k, int32_t m_chunks, size_t* bytes) {
    if (!bytes) return MORE_ERR_INVALID_ARG;
    more_status s = check_lowrank(T, h, r, M, k, m_chunks);
    if (s != MORE_OK) return s;
    if (T == 0) {
        *bytes = 0;
        return MORE_OK;
    }
    if (more::wide_route_needed(r, k)) {
        more::WidePlan w;
        if (!more::wide_make_plan(T, h, r, M, k, &w)) return MORE_ERR_INVALID_ARG;
        *bytes = w.workspace_bytes;
        return MORE_OK;
    }
    more::LowrankPlan p;
    if (!more::lowrank_make_plan(T, h, r, M, k, m_chunks, &p)) return MORE_ERR_INVALID_ARG;
    *bytes = p.workspace_bytes;
    return MORE_OK;
}

more_status more_route_lowrank_workspace_size(int64_t T, int32_t h, int32_t r, int32_t M,
                                              int32_t k, size_t* bytes) {
    return more_route_lowrank_workspace_size_ex(T, h, r, M, k, 0, bytes);
}

more_status more_route_lowrank_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                    int32_t* m_chunks) {
    if (!m_chunks) return MORE_ERR_INVALID_ARG;
    more_status s = check_lowrank(T, h, r, M, k, 0);
    if (s != MORE_OK) return s;
    if (more::wide_route_needed(r, k)) {
        *m_chunks = 0;
        return MORE_OK;
    }
    more::LowrankPlan p;
    if (!more::lowrank_make_plan(T > 0 ? T : 1, h, r, M, k, 0, &p)) return MORE_ERR_INVALID_ARG;
    *m_chunks = p.fused || p.single_pass ? 0 : p.chunks;
    return MORE_OK;
}

more_status more_route_lowrank_route(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                     int32_t* route) {
    if (!route) return MORE_ERR_INVALID_ARG;
    more_status s = check_lowrank(T, h, r, M, k, 0);
    if (s != MORE_OK) return s;
    if (more::wide_route_needed(r, k)) {
        *route = MORE_ROUTE_WIDE;
        return MORE_OK;
    }
    more::LowrankPlan p;
    if (!more::lowrank_make_plan(T > 0 ? T : 1, h, r, M, k, 0, &p)) return MORE_ERR_INVALID_ARG;
    *route = p.single_pass ? MORE_ROUTE_SINGLE_PASS
             : p.local     ? MORE_ROUTE_FUSED_LOCAL
             : p.fused     ? MORE_ROUTE_FUSED
                           : MORE_ROUTE_RESIDENT;
    return MORE_OK;
}

more_status more_route_lowrank_ex(const uint16_t* x, const uint16_t* R1t, const uint16_t* R2t,
                                  int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                  int32_t m_chunks, int32_t* idx, float* gate, float* topval,
                                  int32_t* counts, void* workspace, size_t workspace_bytes,
                                  void* stream) {
    // the token-sized buffers of an empty batch may be NULL (an empty tensor has no storage)
    if (!R1t || !R2t || (T != 0 && (!x || !idx || !gate))) return MORE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(R1t, 16) || !aligned(R2t, 16) || !aligned(idx, 4) ||
        !aligned(gate, 4) || !aligned(topval, 4) || !aligned(counts, 4) || !aligned(workspace, 16))
        return MORE_ERR_INVALID_ARG;
    more_status s = check_lowrank(T, h, r, M, k, m_chunks);
    if (s != MORE_OK) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (T == 0) {
        if (counts) return from_hip(more::histogram_launch(idx, 0, M, counts, st));
        return MORE_OK;
    }
    if (more::wide_route_needed(r, k)) {
        more::WidePlan w;
        if (!more::wide_make_plan(T, h, r, M, k, &w)) return MORE_ERR_INVALID_ARG;
        if (!workspace || workspace_bytes < w.workspace_bytes) return MORE_ERR_WORKSPACE;
        if (more::wide_launch(w, x, R1t, R2t, T, h, r, M, k, idx, gate, topval, workspace, st) !=
            hipSuccess)
            return MORE_ERR_HIP;
        if (counts) return from_hip(more::histogram_launch(idx, T * (int64_t)k, M, counts, st));
        return MORE_OK;
    }
    more::LowrankPlan p;
    if (!more::lowrank_make_plan(T, h, r, M, k, m_chunks, &p)) return MORE_ERR_INVALID_ARG;
    if (p.workspace_bytes > 0 && (!workspace || workspace_bytes < p.workspace_bytes))
        return MORE_ERR_WORKSPACE;
    hipError_t e = more::lowrank_launch(p, x, R1t, R2t, T, h, r, M, k, idx, gate, topval,
                                        counts, workspace, st);
    if (e != hipSuccess) return MORE_ERR_HIP;
    if (counts)  // cleared by the routing launch above
        return from_hip(more::histogram_launch(idx, T * (int64_t)k, M, counts, st, true));
    return MORE_OK;
}

more_status more_route_lowrank(const uint16_t* x, const uint16_t* R1t, const uint16_t* R2t,
                               int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                               int32_t* idx, float* gate, float* topval, int32_t* counts,
                               void* workspace, size_t workspace_bytes, void* stream) {
    return more_route_lowrank_ex(x, R1t, R2t, T, h, r, M, k, 0, idx, gate, topval, counts,
                                 workspace, workspace_bytes, stream);
}

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// Route plan and statistics plan of a training call; the workspace holds the route's workspace
// followed by the statistics'.
static bool train_plans(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                        more::LowrankPlan* lp, more::StatsPlan* sp, size_t* bytes) {
    if (!more::lowrank_make_plan(T, h, r, M, k, 0, lp)) return false;
    if (!more::stats_make_plan(T, h, r, M, k, lp->local != 0, sp)) return false;
    *bytes = align256(lp->workspace_bytes) + sp->workspace_bytes;
    return true;
}

more_status more_route_lowrank_train_workspace_size(int64_t T, int32_t h, int32_t r, int32_t M,
                                                    int32_t k, size_t* bytes) {
    if (!bytes) return MORE_ERR_INVALID_ARG;
    more_status s = check_lowrank(T, h, r, M, k, 0, true);
    if (s != MORE_OK) return s;
    if (T == 0) {
        *bytes = 0;
        return MORE_OK;
    }
    more::LowrankPlan lp;
    more::StatsPlan sp;
    if (!train_plans(T, h, r, M, k, &lp, &sp, bytes)) return MORE_ERR_INVALID_ARG;
    return MORE_OK;
}

more_status more_route_lowrank_train(const uint16_t* x, const uint16_t* R1t, const uint16_t* R2t,
                                     int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                     int32_t* idx, float* gate, float* topval, int32_t* counts,
                                     float* m, float* Z, float* psum, void* workspace,
                                     size_t workspace_bytes, void* stream) {
    if (!R1t || !R2t || !psum || (T != 0 && (!x || !idx || !gate || !m || !Z)))
        return MORE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(R1t, 16) || !aligned(R2t, 16) || !aligned(idx, 4) ||
        !aligned(gate, 4) || !aligned(topval, 4) || !aligned(counts, 4) || !aligned(m, 4) ||
        !aligned(Z, 4) || !aligned(psum, 4) || !aligned(workspace, 256))
        return MORE_ERR_INVALID_ARG;
    more_status s = check_lowrank(T, h, r, M, k, 0, true);
    if (s != MORE_OK) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (T == 0) {
        if (counts) {
            s = from_hip(more::histogram_launch(idx, 0, M, counts, st));
            if (s != MORE_OK) return s;
        }
        return from_hip(more::stats_zero_psum(psum, M, st));
    }
    more::LowrankPlan lp;
    more::StatsPlan sp;
    size_t need = 0;
    if (!train_plans(T, h, r, M, k, &lp, &sp, &need)) return MORE_ERR_INVALID_ARG;
    if (!workspace || workspace_bytes < need) return MORE_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);
    char* sws = ws + align256(lp.workspace_bytes);
    float* tv = topval ? topval : reinterpret_cast<float*>(sws + sp.off_tv);
    hipError_t e = more::lowrank_launch(lp, x, R1t, R2t, T, h, r, M, k, idx, gate, tv, counts,
                                        lp.local ? nullptr : ws, st);
    if (e != hipSuccess) return MORE_ERR_HIP;
    if (counts) {
        e = more::histogram_launch(idx, T * (int64_t)k, M, counts, st, true);
        if (e != hipSuccess) return MORE_ERR_HIP;
    }
    more::StatsArgs a;
    a.x = x;
    a.R1t = R1t;
    a.R2t = R2t;
    a.z = lp.local ? nullptr : reinterpret_cast<const float*>(ws + lp.off_z);
    a.mtop = tv;
    a.ks = k;
    a.T = (int32_t)T;
    a.h = h;
    a.r = r;
    a.M = M;
    a.m = m;
    a.Z = Z;
    a.psum = psum;
    return from_hip(more::stats_launch(sp, a, sws, st));
}

more_status more_route_lowrank_backward_workspace_size(int64_t T, int32_t h, int32_t r,
                                                       int32_t M, int32_t k, int32_t balance,
                                                       size_t* bytes) {
    if (!bytes || r <= 0) return MORE_ERR_INVALID_ARG;
    more_status s = check_common(T, h, M, k);
    if (s != MORE_OK) return s;
    if (!rank_supported(r)) return MORE_ERR_UNSUPPORTED;
    if (T == 0) {
        *bytes = 0;
        return MORE_OK;
    }
    more::BackwardPlan p;
    if (!more::backward_make_plan(T, h, r, M, k, balance != 0, &p)) return MORE_ERR_INVALID_ARG;
    *bytes = p.workspace_bytes;
    return MORE_OK;
}

more_status more_route_lowrank_backward(const uint16_t* x, const uint16_t* R1t,
                                        const uint16_t* R2t, int64_t T, int32_t h, int32_t r,
                                        int32_t M, int32_t k, const int32_t* idx,
                                        const float* dtop, const float* pbar, const float* m,
                                        const float* Z, float* dx, float* dR1t, float* dR2t,
                                        void* workspace, size_t workspace_bytes, void* stream) {
    if (!R1t || !R2t || !dR1t || !dR2t || (T != 0 && (!x || !idx || !dtop || !dx)) ||
        (T != 0 && pbar && (!m || !Z)))
        return MORE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(R1t, 16) || !aligned(R2t, 16) || !aligned(idx, 4) ||
        !aligned(dtop, 4) || !aligned(pbar, 4) || !aligned(m, 4) || !aligned(Z, 4) ||
        !aligned(dx, 4) || !aligned(dR1t, 4) || !aligned(dR2t, 4) || !aligned(workspace, 256))
        return MORE_ERR_INVALID_ARG;
    if (r <= 0) return MORE_ERR_INVALID_ARG;
    more_status s = check_common(T, h, M, k);
    if (s != MORE_OK) return s;
    if (!rank_supported(r)) return MORE_ERR_UNSUPPORTED;
    more::BackwardPlan p;
    if (!more::backward_make_plan(T, h, r, M, k, pbar != nullptr, &p)) return MORE_ERR_INVALID_ARG;
    if (T != 0 && (!workspace || workspace_bytes < p.workspace_bytes)) return MORE_ERR_WORKSPACE;
    more::BackwardArgs a;
    a.x = x;
    a.R1t = R1t;
    a.R2t = R2t;
    a.T = (int32_t)T;
    a.h = h;
    a.r = r;
    a.M = M;
    a.k = k;
    a.idx = idx;
    a.dtop = dtop;
    a.pbar = pbar;
    a.m = m;
    a.Z = Z;
    a.dx = dx;
    a.dR1t = dR1t;
    a.dR2t = dR2t;
    return from_hip(more::backward_launch(p, a, workspace, static_cast<hipStream_t>(stream)));
}

more_status more_route_fullrank_workspace_size(int64_t T, int32_t h, int32_t M, int32_t k,
                                               int32_t logit_bits, size_t* bytes) {
    if (!bytes) return MORE_ERR_INVALID_ARG;
    more_status s = check_common(T, h, M, k);
    if (s != MORE_OK) return s;
    if (logit_bits != 16 && logit_bits != 32) return MORE_ERR_INVALID_ARG;
    if (T == 0) {
        *bytes = 0;
        return MORE_OK;
    }
    more::FullrankPlan p;
    more::fullrank_make_plan(T, h, M, k, logit_bits, &p);
    *bytes = p.workspace_bytes;
    return MORE_OK;
}

more_status more_route_fullrank(const uint16_t* x, const uint16_t* Wt, int64_t T, int32_t h,
                                int32_t M, int32_t k, int32_t logit_bits, int32_t* idx,
                                float* gate, float* topval, void* workspace,
                                size_t workspace_bytes, void* stream) {
    if (!x || !Wt || !idx || !gate) return MORE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(Wt, 16) || !aligned(idx, 4) || !aligned(gate, 4) ||
        !aligned(topval, 4) || !aligned(workspace, 256))
        return MORE_ERR_INVALID_ARG;
    more_status s = check_common(T, h, M, k);
    if (s != MORE_OK) return s;
    if (logit_bits != 16 && logit_bits != 32) return MORE_ERR_INVALID_ARG;
    if (T == 0) return MORE_OK;
    more::FullrankPlan p;
    more::fullrank_make_plan(T, h, M, k, logit_bits, &p);
    if (!workspace || workspace_bytes < p.workspace_bytes) return MORE_ERR_WORKSPACE;
    int blas = 0;
    hipError_t e = more::fullrank_launch(p, x, Wt, T, h, M, k, idx, gate, topval, workspace,
                                         static_cast<hipStream_t>(stream), &blas);
    return from_hip(e);
}

more_status more_route_fullrank_fused_workspace_size(int64_t T, int32_t h, int32_t M, int32_t k,
                                                     size_t* bytes) {
    if (!bytes) return MORE_ERR_INVALID_ARG;
    more_status s = check_common(T, h, M, k);
    if (s != MORE_OK) return s;
    more::FusedFullrankPlan p;
    if (!more::fullrank_fused_make_plan(T > 0 ? T : 1, h, M, k, &p)) return MORE_ERR_UNSUPPORTED;
    *bytes = T == 0 ? 0 : p.workspace_bytes;
    return MORE_OK;
}

more_status more_route_fullrank_fused(const uint16_t* x, const uint16_t* Wt, int64_t T, int32_t h,
                                      int32_t M, int32_t k, int32_t* idx, float* gate,
                                      float* topval, void* workspace, size_t workspace_bytes,
                                      void* stream) {
    if (!Wt || (T != 0 && (!x || !idx || !gate))) return MORE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(Wt, 16) || !aligned(idx, 4) || !aligned(gate, 4) ||
        !aligned(topval, 4) || !aligned(workspace, 16))
        return MORE_ERR_INVALID_ARG;
    size_t need = 0;
    more_status s = more_route_fullrank_fused_workspace_size(T, h, M, k, &need);
    if (s != MORE_OK) return s;
    if (T == 0) return MORE_OK;
    if (need > 0 && (!workspace || workspace_bytes < need)) return MORE_ERR_WORKSPACE;
    more::FusedFullrankPlan p;
    more::fullrank_fused_make_plan(T, h, M, k, &p);
    return from_hip(more::fullrank_fused_launch(p, x, Wt, T, h, M, k, idx, gate, topval, workspace,
                                                static_cast<hipStream_t>(stream)));
}

more_status more_dispatch_sort_workspace_size(int64_t T, int32_t k, int32_t M, size_t* bytes) {
    if (!bytes || T < 0 || k < 1 || M < 1) return MORE_ERR_INVALID_ARG;
    if (T > kMaxT || M >= kMaxM || T * (int64_t)k > kMaxT) return MORE_ERR_UNSUPPORTED;
    *bytes = more::dispatch_workspace_bytes(T * (int64_t)k);
    return MORE_OK;
}

more_status more_dispatch_sort(const int32_t* idx, int64_t T, int32_t k, int32_t M,
                               int32_t* offsets, int32_t* sorted, void* workspace,
                               size_t workspace_bytes, void* stream) {
    if (!offsets || (T > 0 && (!idx || !sorted))) return MORE_ERR_INVALID_ARG;
    if (!aligned(idx, 4) || !aligned(offsets, 4) || !aligned(sorted, 4) || !aligned(workspace, 256))
        return MORE_ERR_INVALID_ARG;
    size_t need = 0;
    more_status s = more_dispatch_sort_workspace_size(T, k, M, &need);
    if (s != MORE_OK) return s;
    if (need > 0 && (!workspace || workspace_bytes < need)) return MORE_ERR_WORKSPACE;
    return from_hip(more::dispatch_launch(idx, T * (int64_t)k, M, offsets, sorted, workspace,
                                          static_cast<hipStream_t>(stream)));
}

more_status more_expert_histogram(const int32_t* idx, int64_t T, int32_t k, int32_t M,
                                  int32_t* counts, void* stream) {
    if (!counts || (!idx && T > 0)) return MORE_ERR_INVALID_ARG;
    if (!aligned(idx, 4) || !aligned(counts, 4)) return MORE_ERR_INVALID_ARG;
    if (T < 0 || k < 1 || M < 1) return MORE_ERR_INVALID_ARG;
    if (T > kMaxT || M > kMaxM) return MORE_ERR_UNSUPPORTED;
    return from_hip(more::histogram_launch(idx, T * (int64_t)k, M, counts,
                                           static_cast<hipStream_t>(stream)));
}

}  // extern "C"
