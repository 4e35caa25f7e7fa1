// Gradients of the SpinGTP forward (spingtp_backward).
//
// For y[k3] = sum T[k1,k2,k3] x1[k1] x2[k2] and a loss gradient g = dL/dy, the
// chain rule gives gx1[k1] = sum T[k1,k2,k3] x2[k2] g[k3] (and gx2 likewise).
// Conjugating the Gaunt integral (Sec. 3.2 eq. generalized_gaunt) with the
// conjugation relation of App. A.1 turns this into another SpinGTP product:
// T[k1,k2,k3] = sum_j T'[k3,j,k1] J[j,k2], with T' the tensor of degrees
// (Lout, L2, L1) and J the real matrix of conjugation on real-basis coefficients.
// So gx1 = SpinGTP'(g, J x2) and gx2 = SpinGTP''(g, J x1).  For L1 = L2 = Lout
// both are launches of the plan's own forward kernel (the instantiation whose
// input-2 lanes read the second copy of the m = 0 mixing of the |s| = 1 sectors)
// on the plan's backward tables, where that copy absorbs J (J moves no other
// slots); no copy of J x is made.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace {

bool misaligned(const void* p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) != 0;
}

}  // namespace

extern "C" spingtp_status spingtp_backward(spingtp_plan plan, const void* x1, const void* x2, const void* grad_out,
                                           void* grad_x1, void* grad_x2, int64_t N, int64_t C, void* stream) {
    if (plan == nullptr || N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_tab_bwd == nullptr) return SPINGTP_ERR_UNSUPPORTED;
    if (N == 0 || C == 0 || (grad_x1 == nullptr && grad_x2 == nullptr)) return SPINGTP_OK;
    if (misaligned(grad_x1) || misaligned(grad_x2)) return SPINGTP_ERR_INVALID_ARG;
    // run_forward checks the rest (sizes, pointers, alignment, device)
    if (grad_x1 != nullptr) {
        const spingtp_status r =
            spingtp::run_forward(plan, plan->kernel, grad_out, x2, grad_x1, N, C, false, stream, plan->d_tab_bwd,
                                 true);
        if (r != SPINGTP_OK) return r;
    }
    if (grad_x2 != nullptr) {
        const spingtp_status r =
            spingtp::run_forward(plan, plan->kernel, grad_out, x1, grad_x2, N, C, false, stream, plan->d_tab_bwd,
                                 true);
        if (r != SPINGTP_OK) return r;
    }
    return SPINGTP_OK;
}
