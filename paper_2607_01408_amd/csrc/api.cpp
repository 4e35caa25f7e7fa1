// C entry points of the forward launches (argument checks, kernel choice of the
// plan, launch on the caller's stream).  The kernels are in forward.hip,
// forward_mfma.hip and forward_pre*.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "internal.h"

spingtp_status spingtp::run_forward(spingtp_plan plan, const spingtp::KernelEntry* k, const void* x1, const void* x2,
                                    void* out, int64_t N, int64_t C, bool shared_x2, void* stream,
                                    const float* tab, bool backward, const uint32_t* aux_override) {
    if (plan == nullptr || N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
    if (N == 0 || C == 0) return SPINGTP_OK;
    if (N > (int64_t{1} << 40) / C) return SPINGTP_ERR_INVALID_ARG;
    if (x1 == nullptr || x2 == nullptr || out == nullptr) return SPINGTP_ERR_INVALID_ARG;
    const auto misaligned = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; };
    if (misaligned(x1) || misaligned(x2) || misaligned(out)) return SPINGTP_ERR_INVALID_ARG;
    if (k == nullptr) return SPINGTP_ERR_UNSUPPORTED;
    const bool bwd_launch = backward && k->family != 5;  // family 5 takes J through its table
    if (bwd_launch && k->launch_bwd == nullptr) return SPINGTP_ERR_UNSUPPORTED;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const uint32_t* aux =
        aux_override != nullptr ? aux_override
                                : (k->family == 5 ? plan->d_pre : (k->family == 6 ? plan->d_dir : plan->d_aux));
    const hipError_t e =
        k->launch_lds != nullptr
            ? k->launch_lds(x1, x2, out, N * C, shared_x2 ? C : 1, aux, plan->dir_lds_floats,
                            static_cast<hipStream_t>(stream))
            : (bwd_launch ? k->launch_bwd : k->launch)(x1, x2, out, N * C, shared_x2 ? C : 1,
                                                       tab != nullptr ? tab : plan->d_tab, aux,
                                                       static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}

extern "C" spingtp_status spingtp_forward(spingtp_plan plan, const void* x1, const void* x2, void* out, int64_t N,
                                          int64_t C, void* stream) {
    return spingtp::run_forward(plan, plan ? plan->kernel : nullptr, x1, x2, out, N, C, false, stream);
}

extern "C" spingtp_status spingtp_forward_v1(spingtp_plan plan, const void* x1, const void* x2, void* out,
                                             int64_t N, int64_t C, void* stream) {
    return spingtp::run_forward(plan, plan ? plan->kernel_v1 : nullptr, x1, x2, out, N, C, true, stream);
}

extern "C" spingtp_status spingtp_forward_v1_weighted(spingtp_plan plan, const void* x1, const void* x2,
                                                      const float* weights, void* out, int64_t N, int64_t C,
                                                      void* stream) {
    if (plan == nullptr) return SPINGTP_ERR_INVALID_ARG;
    // the entry-list kernel unless the plan asks for the precontracted route
    const bool entry_lists = plan->d_bw1w != nullptr && plan->bw1w.lds_shared_fwd > 0 &&
                             !((plan->flags & SPINGTP_V1_PRECONTRACT) && plan->kernel_v1w != nullptr);
    if (plan->kernel_v1w == nullptr && !entry_lists) return SPINGTP_ERR_UNSUPPORTED;
    if (N > 0 && C > 0 && (weights == nullptr || (reinterpret_cast<uintptr_t>(weights) & 3u) != 0))
        return SPINGTP_ERR_INVALID_ARG;
    if (entry_lists) {  // the entry-list kernel (measured faster on the depthwise runtime table's shapes)
        if (N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
        if (N == 0 || C == 0) return SPINGTP_OK;
        if (N > (int64_t{1} << 40) / C) return SPINGTP_ERR_INVALID_ARG;
        if (x1 == nullptr || x2 == nullptr || out == nullptr) return SPINGTP_ERR_INVALID_ARG;
        const auto misaligned = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; };
        if (misaligned(x1) || misaligned(x2) || misaligned(out)) return SPINGTP_ERR_INVALID_ARG;
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
        if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
        const hipError_t e = spingtp::launch_fwd_cw(plan->dtype == SPINGTP_FP32 ? 0 : 1, true, x1, x2, weights, out,
                                                    N, C, plan->bw1w, plan->d_bw1w, static_cast<hipStream_t>(stream));
        return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
    }
    // the weighted precontracted kernel takes the weights in place of the plan tables
    return spingtp::run_forward(plan, plan->kernel_v1w, x1, x2, out, N, C, true, stream, weights, false,
                                plan->d_pre_w);
}

extern "C" spingtp_status spingtp_backward_v1_weighted_workspace_size(spingtp_plan plan, int64_t N, int64_t C,
                                                                      size_t* bytes) {
    if (plan == nullptr || bytes == nullptr || N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_bw1w == nullptr) return SPINGTP_ERR_UNSUPPORTED;
    if (N > 0 && C > 0 && N > (int64_t{1} << 40) / C) return SPINGTP_ERR_INVALID_ARG;
    *bytes = spingtp::bw1w_workspace_floats(N, C, plan->bw1w) * sizeof(float);
    return SPINGTP_OK;
}

extern "C" spingtp_status spingtp_backward_v1_weighted(spingtp_plan plan, const void* x1, const void* x2,
                                                       const float* weights, const void* grad_out, void* grad_x1,
                                                       void* grad_x2, float* grad_weights, void* workspace,
                                                       size_t workspace_bytes, int64_t N, int64_t C, void* stream) {
    size_t need = 0;
    const spingtp_status st = spingtp_backward_v1_weighted_workspace_size(plan, N, C, &need);
    if (st != SPINGTP_OK) return st;
    if (N == 0 && C == 0) return SPINGTP_OK;  // every output is empty
    const auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
    // every array with elements must be present; the unit arrays are empty when C = 0
    if ((N > 0 && (x2 == nullptr || grad_x2 == nullptr)) ||
        (N > 0 && C > 0 && (x1 == nullptr || grad_out == nullptr || grad_x1 == nullptr)) ||
        (C > 0 && (weights == nullptr || grad_weights == nullptr)))
        return SPINGTP_ERR_INVALID_ARG;
    if (misaligned(x1, 16) || misaligned(x2, 16) || misaligned(grad_out, 16) || misaligned(grad_x1, 16) ||
        misaligned(grad_x2, 16) || misaligned(weights, 4) || misaligned(grad_weights, 4) || misaligned(workspace, 4))
        return SPINGTP_ERR_INVALID_ARG;
    if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return SPINGTP_ERR_INVALID_ARG;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const hipError_t e = spingtp::launch_bwd_v1w(
        plan->dtype == SPINGTP_FP32 ? 0 : 1, true, x1, x2, weights, grad_out, grad_x1, grad_x2, grad_weights,
        static_cast<float*>(workspace), N, C, plan->bw1w, plan->d_bw1w, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}

extern "C" spingtp_status spingtp_forward_weighted(spingtp_plan plan, const void* x1, const void* x2,
                                                   const float* weights, void* out, int64_t N, int64_t C,
                                                   void* stream) {
    if (plan == nullptr || N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_bw1w == nullptr || plan->bw1w.lds_unit_fwd == 0) return SPINGTP_ERR_UNSUPPORTED;
    if (N == 0 || C == 0) return SPINGTP_OK;
    if (N > (int64_t{1} << 40) / C) return SPINGTP_ERR_INVALID_ARG;
    if (x1 == nullptr || x2 == nullptr || out == nullptr || weights == nullptr) return SPINGTP_ERR_INVALID_ARG;
    const auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
    if (misaligned(x1, 16) || misaligned(x2, 16) || misaligned(out, 16) || misaligned(weights, 4))
        return SPINGTP_ERR_INVALID_ARG;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const hipError_t e = spingtp::launch_fwd_cw(plan->dtype == SPINGTP_FP32 ? 0 : 1, false, x1, x2, weights, out, N,
                                                C, plan->bw1w, plan->d_bw1w, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}

extern "C" spingtp_status spingtp_backward_weighted_workspace_size(spingtp_plan plan, int64_t N, int64_t C,
                                                                   size_t* bytes) {
    if (plan == nullptr || bytes == nullptr || N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_bw1w == nullptr || plan->bw1w.lds_unit_bwd == 0) return SPINGTP_ERR_UNSUPPORTED;
    if (N > 0 && C > 0 && N > (int64_t{1} << 40) / C) return SPINGTP_ERR_INVALID_ARG;
    *bytes = spingtp::bwcw_workspace_floats(N, C, plan->bw1w) * sizeof(float);
    return SPINGTP_OK;
}

extern "C" spingtp_status spingtp_backward_weighted(spingtp_plan plan, const void* x1, const void* x2,
                                                    const float* weights, const void* grad_out, void* grad_x1,
                                                    void* grad_x2, float* grad_weights, void* workspace,
                                                    size_t workspace_bytes, int64_t N, int64_t C, void* stream) {
    size_t need = 0;
    const spingtp_status st = spingtp_backward_weighted_workspace_size(plan, N, C, &need);
    if (st != SPINGTP_OK) return st;
    if (C == 0) return SPINGTP_OK;  // every output is empty
    const auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
    if ((N > 0 && (x1 == nullptr || x2 == nullptr || grad_out == nullptr || grad_x1 == nullptr ||
                   grad_x2 == nullptr)) ||
        weights == nullptr || grad_weights == nullptr)
        return SPINGTP_ERR_INVALID_ARG;
    if (misaligned(x1, 16) || misaligned(x2, 16) || misaligned(grad_out, 16) || misaligned(grad_x1, 16) ||
        misaligned(grad_x2, 16) || misaligned(weights, 4) || misaligned(grad_weights, 4) || misaligned(workspace, 4))
        return SPINGTP_ERR_INVALID_ARG;
    if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return SPINGTP_ERR_INVALID_ARG;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const hipError_t e = spingtp::launch_bwd_v1w(
        plan->dtype == SPINGTP_FP32 ? 0 : 1, false, x1, x2, weights, grad_out, grad_x1, grad_x2, grad_weights,
        static_cast<float*>(workspace), N, C, plan->bw1w, plan->d_bw1w, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}

extern "C" spingtp_status spingtp_forward_depthwise(spingtp_plan plan, const void* x1, const void* x2,
                                                    const float* weights, void* out, int64_t N, int64_t C, int64_t V,
                                                    void* stream) {
    if (plan == nullptr || N < 0 || C < 0 || V < 1) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_bw1w == nullptr || plan->bw1w.lds_shared_fwd == 0) return SPINGTP_ERR_UNSUPPORTED;
    if (N == 0 || C == 0) return SPINGTP_OK;
    if (N > (int64_t{1} << 40) / C || V > (int64_t{1} << 20)) return SPINGTP_ERR_INVALID_ARG;
    if (x1 == nullptr || x2 == nullptr || out == nullptr || weights == nullptr) return SPINGTP_ERR_INVALID_ARG;
    const auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
    if (misaligned(x1, 16) || misaligned(x2, 16) || misaligned(out, 16) || misaligned(weights, 4))
        return SPINGTP_ERR_INVALID_ARG;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const int64_t n2 = plan->bw1w.nc2, elem = plan->dtype == SPINGTP_FP32 ? 4 : 2;
    const int64_t wslice = C * plan->bw1w.np;
    // up to kFwdCwMaxNv channels per launch, as many as the LDS holds without fewer
    // workgroups per CU than one channel gets (at least two); later launches add
    // into out, in channel order
    const int lds1 = spingtp::fwd_cw_lds_floats(plan->bw1w, 1);
    const int per_cu1 = std::min(2, spingtp::kBw1wMaxLdsFloats / std::max(lds1, 1));
    int nv_max = 1;
    while (nv_max < spingtp::kFwdCwMaxNv &&
           spingtp::kBw1wMaxLdsFloats / spingtp::fwd_cw_lds_floats(plan->bw1w, nv_max + 1) >= per_cu1)
        ++nv_max;
    for (int64_t v = 0; v < V;) {
        const int nv = static_cast<int>(std::min<int64_t>(nv_max, V - v));
        const hipError_t e = spingtp::launch_fwd_cw(
            plan->dtype == SPINGTP_FP32 ? 0 : 1, true, x1, static_cast<const char*>(x2) + v * n2 * elem,
            weights + v * wslice, out, N, C, plan->bw1w, plan->d_bw1w, static_cast<hipStream_t>(stream), V * n2,
            v > 0, nv, n2, wslice);
        if (e != hipSuccess) return SPINGTP_ERR_HIP;
        v += nv;
    }
    return SPINGTP_OK;
}

extern "C" spingtp_status spingtp_backward_depthwise_workspace_size(spingtp_plan plan, int64_t N, int64_t C,
                                                                    int64_t V, size_t* bytes) {
    if (V < 1) return SPINGTP_ERR_INVALID_ARG;
    return spingtp_backward_v1_weighted_workspace_size(plan, N, C, bytes);  // reused by every channel v
}

extern "C" spingtp_status spingtp_backward_depthwise(spingtp_plan plan, const void* x1, const void* x2,
                                                     const float* weights, const void* grad_out, void* grad_x1,
                                                     void* grad_x2, float* grad_weights, void* workspace,
                                                     size_t workspace_bytes, int64_t N, int64_t C, int64_t V,
                                                     void* stream) {
    size_t need = 0;
    if (V < 1 || V > (int64_t{1} << 20)) return SPINGTP_ERR_INVALID_ARG;
    const spingtp_status st = spingtp_backward_v1_weighted_workspace_size(plan, N, C, &need);
    if (st != SPINGTP_OK) return st;
    if (N == 0 && C == 0) return SPINGTP_OK;
    const auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
    if ((N > 0 && (x2 == nullptr || grad_x2 == nullptr)) ||
        (N > 0 && C > 0 && (x1 == nullptr || grad_out == nullptr || grad_x1 == nullptr)) ||
        (C > 0 && (weights == nullptr || grad_weights == nullptr)))
        return SPINGTP_ERR_INVALID_ARG;
    if (misaligned(x1, 16) || misaligned(x2, 16) || misaligned(grad_out, 16) || misaligned(grad_x1, 16) ||
        misaligned(grad_x2, 16) || misaligned(weights, 4) || misaligned(grad_weights, 4) || misaligned(workspace, 4))
        return SPINGTP_ERR_INVALID_ARG;
    if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return SPINGTP_ERR_INVALID_ARG;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const int64_t n2 = plan->bw1w.nc2, elem = plan->dtype == SPINGTP_FP32 ? 4 : 2;
    const int64_t wslice = C * plan->bw1w.np;
    for (int64_t v = 0; v < V; ++v) {  // grad_x1 sums the channels' terms in order; the rest is per channel
        const hipError_t e = spingtp::launch_bwd_v1w(
            plan->dtype == SPINGTP_FP32 ? 0 : 1, true, x1, static_cast<const char*>(x2) + v * n2 * elem,
            weights + v * wslice, grad_out, grad_x1, static_cast<char*>(grad_x2) + v * n2 * elem,
            grad_weights + v * wslice, static_cast<float*>(workspace), N, C, plan->bw1w, plan->d_bw1w,
            static_cast<hipStream_t>(stream), V * n2, v > 0);
        if (e != hipSuccess) return SPINGTP_ERR_HIP;
    }
    return SPINGTP_OK;
}
