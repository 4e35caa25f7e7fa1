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
// slots); no copy of J x is made.  Plans on the direct sparse-tensor kernel, and
// non-square plans whose transposed degrees have no Fourier kernel, run the two
// gradients as that kernel on the tensor's other two roles (entries of T listed
// by k1 and by k2), which needs no conjugation.  The shared-x2 form
// (spingtp_backward_v1) is at the end of the file.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "internal.h"

namespace {

bool misaligned(const void* p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) != 0;
}

}  // namespace

extern "C" spingtp_status spingtp_backward(spingtp_plan plan, const void* x1, const void* x2, const void* grad_out,
                                           void* grad_x1, void* grad_x2, int64_t N, int64_t C, void* stream) {
    if (plan == nullptr || N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_tab_bwd == nullptr && plan->d_dir_b1 == nullptr) return SPINGTP_ERR_UNSUPPORTED;
    if (N == 0 || C == 0 || (grad_x1 == nullptr && grad_x2 == nullptr)) return SPINGTP_OK;
    if (misaligned(grad_x1) || misaligned(grad_x2)) return SPINGTP_ERR_INVALID_ARG;
    // run_forward checks the rest (sizes, pointers, alignment, device)
    if (plan->d_tab_bwd == nullptr) {  // the direct kernel on the gradient roles of T
        if (grad_x1 != nullptr) {
            const spingtp_status r = spingtp::run_forward(plan, plan->kernel_dir, grad_out, x2, grad_x1, N, C, false,
                                                          stream, nullptr, false, plan->d_dir_b1);
            if (r != SPINGTP_OK) return r;
        }
        if (grad_x2 != nullptr)
            return spingtp::run_forward(plan, plan->kernel_dir, grad_out, x1, grad_x2, N, C, false, stream, nullptr,
                                        false, plan->d_dir_b2);
        return SPINGTP_OK;
    }
    if (grad_x1 != nullptr) {
        const spingtp_status r =
            spingtp::run_forward(plan, plan->kernel, grad_out, x2, grad_x1, N, C, false, stream, plan->d_tab_bwd,
                                 true, plan->deg_bwd(1));
        if (r != SPINGTP_OK) return r;
    }
    if (grad_x2 != nullptr) {
        const spingtp_status r =
            spingtp::run_forward(plan, plan->kernel, grad_out, x1, grad_x2, N, C, false, stream, plan->d_tab_bwd,
                                 true, plan->deg_bwd(2));
        if (r != SPINGTP_OK) return r;
    }
    return SPINGTP_OK;
}

// ---------------------------------------------------------------------------
// Edge input shared by the channels of an edge (spingtp_forward_v1).
//   grad_x1[n,c] = SpinGTP'(g[n,c], J x2[n])                 (x2 shared: the v1 route)
//   grad_x2[n]   = sum_c SpinGTP''(g[n,c], J x1[n,c])          (per unit, then summed)
// The per-unit products of grad_x2 go to the caller's workspace [N][C][NC2] and a
// reduction kernel sums them over the channels in a fixed order.
// ---------------------------------------------------------------------------
namespace {

constexpr int kSumThreads = 256;

template <typename T>
__device__ __forceinline__ float load_f32(const T* p);
template <>
__device__ __forceinline__ float load_f32<float>(const float* p) {
    return *p;
}
template <>
__device__ __forceinline__ float load_f32<uint16_t>(const uint16_t* p) {  // bf16 bits
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
}
template <typename T>
__device__ __forceinline__ T store_f32(float v);
template <>
__device__ __forceinline__ float store_f32<float>(float v) {
    return v;
}
template <>
__device__ __forceinline__ uint16_t store_f32<uint16_t>(float v) {  // round to nearest even
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7f800000u) == 0x7f800000u) return static_cast<uint16_t>((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// out[n][k] = sum_{c < C} in[n][c][k], fp32 sums in channel order; one thread per (n, k).
template <typename T>
__global__ __launch_bounds__(kSumThreads) void spingtp_sum_channels_kernel(const T* __restrict__ in,
                                                                          T* __restrict__ out, int64_t N,
                                                                          int64_t C, int nc) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kSumThreads + threadIdx.x;
    if (i >= N * nc) return;
    const int64_t n = i / nc;
    const int k = static_cast<int>(i - n * nc);
    const T* __restrict__ p = in + n * C * nc + k;
    float acc = 0.f;
    for (int64_t c = 0; c < C; ++c) acc += load_f32<T>(p + c * nc);
    out[i] = store_f32<T>(acc);
}

hipError_t launch_sum_channels(const void* in, void* out, int64_t N, int64_t C, int nc, int dtype,
                               hipStream_t stream) {
    const int64_t blocks = (N * nc + kSumThreads - 1) / kSumThreads;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    if (dtype == SPINGTP_FP32)
        hipLaunchKernelGGL(spingtp_sum_channels_kernel<float>, dim3(static_cast<unsigned>(blocks)), dim3(kSumThreads),
                           0, stream, static_cast<const float*>(in), static_cast<float*>(out), N, C, nc);
    else
        hipLaunchKernelGGL(spingtp_sum_channels_kernel<uint16_t>, dim3(static_cast<unsigned>(blocks)),
                           dim3(kSumThreads), 0, stream, static_cast<const uint16_t*>(in),
                           static_cast<uint16_t*>(out), N, C, nc);
    return hipGetLastError();
}

int64_t row_length(const spingtp_plan_s* p) {
    return static_cast<int64_t>(p->n_spins) * (p->L2 + 1) * (p->L2 + 1);
}

}  // namespace

extern "C" spingtp_status spingtp_backward_v1_workspace_size(spingtp_plan plan, int64_t N, int64_t C,
                                                             size_t* bytes) {
    if (plan == nullptr || bytes == nullptr || N < 0 || C < 0) return SPINGTP_ERR_INVALID_ARG;
    if ((plan->d_tab_bwd == nullptr || plan->kernel == nullptr) && plan->d_dir_b1 == nullptr)
        return SPINGTP_ERR_UNSUPPORTED;
    if (N > 0 && C > 0 && N > (int64_t{1} << 40) / C) return SPINGTP_ERR_INVALID_ARG;
    const size_t elem = plan->dtype == SPINGTP_FP32 ? 4 : 2;
    *bytes = static_cast<size_t>(N) * static_cast<size_t>(C) * static_cast<size_t>(row_length(plan)) * elem;
    return SPINGTP_OK;
}

extern "C" spingtp_status spingtp_backward_v1(spingtp_plan plan, const void* x1, const void* x2,
                                              const void* grad_out, void* grad_x1, void* grad_x2, void* workspace,
                                              size_t workspace_bytes, int64_t N, int64_t C, void* stream) {
    size_t need = 0;
    const spingtp_status st = spingtp_backward_v1_workspace_size(plan, N, C, &need);
    if (st != SPINGTP_OK) return st;
    if (N == 0 || (grad_x1 == nullptr && grad_x2 == nullptr)) return SPINGTP_OK;
    if (misaligned(grad_x1) || misaligned(grad_x2)) return SPINGTP_ERR_INVALID_ARG;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (C == 0) {  // no channels: grad_x2 is an empty sum, written as zeros
        if (grad_x2 == nullptr) return SPINGTP_OK;
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
        if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
        return launch_sum_channels(nullptr, grad_x2, N, 0, static_cast<int>(row_length(plan)), plan->dtype, s) ==
                       hipSuccess
                   ? SPINGTP_OK
                   : SPINGTP_ERR_HIP;
    }
    if (grad_x1 != nullptr) {
        const spingtp::KernelEntry* k = plan->kernel_v1;
        spingtp_status r;
        if (k != nullptr && k->family == 5 && plan->d_pre_bwd != nullptr) {
            r = spingtp::run_forward(plan, k, grad_out, x2, grad_x1, N, C, true, stream, nullptr, true,
                                     plan->d_pre_bwd);
        } else if (plan->d_tab_bwd != nullptr) {  // the Fourier kernel, x2 read once per edge
            const spingtp::KernelEntry* kf = (k != nullptr && k->family != 5) ? k : plan->kernel;
            r = spingtp::run_forward(plan, kf, grad_out, x2, grad_x1, N, C, true, stream, plan->d_tab_bwd, true,
                                     plan->deg_bwd(1));
        } else if (plan->d_dir_b1 != nullptr) {  // the direct kernel, x2 shared by the channels
            r = spingtp::run_forward(plan, plan->kernel_dir, grad_out, x2, grad_x1, N, C, true, stream, nullptr,
                                     false, plan->d_dir_b1);
        } else {
            return SPINGTP_ERR_UNSUPPORTED;
        }
        if (r != SPINGTP_OK) return r;
    }
    if (grad_x2 != nullptr) {
        if (workspace == nullptr || misaligned(workspace) || workspace_bytes < need) return SPINGTP_ERR_INVALID_ARG;
        const spingtp_status r =
            plan->d_tab_bwd != nullptr
                ? spingtp::run_forward(plan, plan->kernel, grad_out, x1, workspace, N, C, false, stream,
                                       plan->d_tab_bwd, true, plan->deg_bwd(2))
                : spingtp::run_forward(plan, plan->kernel_dir, grad_out, x1, workspace, N, C, false, stream,
                                       nullptr, false, plan->d_dir_b2);
        if (r != SPINGTP_OK) return r;
        if (launch_sum_channels(workspace, grad_x2, N, C, static_cast<int>(row_length(plan)), plan->dtype, s) !=
            hipSuccess)
            return SPINGTP_ERR_HIP;
    }
    return SPINGTP_OK;
}

// ---------------------------------------------------------------------------
// spingtp_backward_v1 without a caller workspace: the grad_x2 staging rows live in
// a fixed device array.  Host code never passes the array's name to a kernel (in
// host code it names a host-side stand-in); it uses the device address looked up
// once per device with that device current.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[SPINGTP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kScratchDevices] = {};

// Device address of `scratch` on the current device (looked up on first use).
spingtp_status scratch_address(int device, void** out) {
    if (device < 0 || device >= kScratchDevices) return SPINGTP_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[device] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return SPINGTP_ERR_HIP;
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return SPINGTP_OK;
}

}  // namespace

extern "C" spingtp_status spingtp_backward_v1_noalloc(spingtp_plan plan, const void* x1, const void* x2,
                                                      const void* grad_out, void* grad_x1, void* grad_x2, int64_t N,
                                                      int64_t C, void* stream) {
    size_t need = 0;
    const spingtp_status st = spingtp_backward_v1_workspace_size(plan, N, C, &need);
    if (st != SPINGTP_OK) return st;
    if (grad_x2 != nullptr && need > SPINGTP_NOALLOC_SCRATCH_BYTES) return SPINGTP_ERR_TOO_LARGE;
    void* ws = nullptr;
    if (grad_x2 != nullptr && N > 0 && C > 0) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
        if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
        const spingtp_status sa = scratch_address(cur, &ws);
        if (sa != SPINGTP_OK) return sa;
    }
    return spingtp_backward_v1(plan, x1, x2, grad_out, grad_x1, grad_x2, ws, SPINGTP_NOALLOC_SCRATCH_BYTES, N, C,
                               stream);
}
