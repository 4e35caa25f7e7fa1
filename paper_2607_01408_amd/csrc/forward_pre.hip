// Precontracted SpinGTP for an edge input shared by the channels of an edge
// (edge multiplicity V = 1; paper Sec. 3.4, the precontraction equations, and
// App. E, depthwise mode with V = 1 and unit weights).
//
// With x2 the same for every channel c of edge n, the bilinear map
//   out[n,c,k3] = sum_{k1,k2} T[k1,k2,k3] x1[n,c,k1] x2[n,k2]
// factors into an edge kernel K_n[k1,k3] = sum_{k2} T[k1,k2,k3] x2[n,k2] (built
// once per edge) and a dense product out[n,c,:] = x1[n,c,:] K_n over the
// channels.  T is the real tensor of the operation (Sec. 3.2 eq. generalized_gaunt
// through the real basis of App. C), built on the host in float64 by the plan.
//
// One workgroup of 256 threads per edge.
//  1. The x2 row goes to LDS and the transposed kernel Kt[k3][k1] (16 NT rows of
//     KST = 16 KS + 4 floats, zero padded) is cleared.
//  2. Kernel build: each thread walks its own list of tensor items (laid out
//     [item][thread], so every load is coalesced and independent of the sums),
//     keeps a running sum and stores it when an entry's list ends.  Whole entries
//     belong to one thread: the build is deterministic and needs no atomics.
//  3. Product on the matrix cores, fp32 in and out (v_mfma_f32_16x16x4_f32): each
//     wave takes tiles of 16 channels and forms D[k3][c] = sum_k1 Kt[k3][k1] x1[c][k1]
//     for 16-row strips of k3.  The contraction index of MFMA step (s, j) for lane
//     group g = lane / 16 is k1 = 16 s + 4 g + j, so a lane reads its four Kt values
//     with one 16-byte LDS load and its four x1 values from one 16-byte run of its
//     channel's row; the accumulator of a lane then holds four consecutive k3 of one
//     channel.
// The l = 0 slots of the |s| = 1 sectors are not data: x1 values there are never
// read (taken as 0), and T has no entries for them, so those outputs are written
// as 0 and x2 values there are never used.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.h"
#include "internal.h"

namespace spingtp {
namespace {

template <typename TIO>
__device__ __forceinline__ TIO from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) {
    return v;
}
template <>
__device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) {
    return f32_to_bf16(v);
}

// KS = ceil(NC1 / 16) contraction blocks, NT = ceil(NCO / 16) output strips.
template <typename TIO, int KS, int NT>
__global__ __launch_bounds__(kPreThreads) void spingtp_fwd_pre_kernel(const TIO* __restrict__ x1,
                                                                      const TIO* __restrict__ x2,
                                                                      TIO* __restrict__ out, int64_t C,
                                                                      const uint32_t* __restrict__ aux) {
    constexpr int KST = 16 * KS + 4;
    constexpr int KT_FLOATS = 16 * NT * KST;
    __shared__ __align__(16) float Kt[KT_FLOATS];
    __shared__ float X2[kPreMaxNC];

    const int NC1 = static_cast<int>(aux[0]), NC2 = static_cast<int>(aux[1]), NCO = static_cast<int>(aux[2]);
    const int blk1 = static_cast<int>(aux[3]), ipt = static_cast<int>(aux[6]);
    const int tid = threadIdx.x;
    const int64_t n = blockIdx.x;

    for (int i = tid; i < KT_FLOATS / 4; i += kPreThreads) reinterpret_cast<v4f*>(Kt)[i] = v4f{0.f, 0.f, 0.f, 0.f};
    for (int i = tid; i < NC2; i += kPreThreads) X2[i] = to_f32(x2[n * NC2 + i]);
    __syncthreads();

    {
        const uint32_t* __restrict__ words = aux + kPreHeader + tid;
        const float* __restrict__ vals = reinterpret_cast<const float*>(aux + kPreHeader + ipt * kPreThreads) + tid;
        float acc = 0.f;
        for (int i = 0; i < ipt; i += 8) {  // ipt is a multiple of 8
            uint32_t w[8];
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                w[j] = words[(i + j) * kPreThreads];
                v[j] = vals[(i + j) * kPreThreads];
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                acc = fmaf(v[j], X2[(w[j] >> 16) & 0xffu], acc);
                if (w[j] >> 24) {
                    Kt[w[j] & 0xffffu] = acc;
                    acc = 0.f;
                }
            }
        }
    }
    __syncthreads();

    const int lane = tid & 63, col = lane & 15, g = lane >> 4;
    const int64_t tiles = (C + 15) / 16;
    const TIO* __restrict__ xe = x1 + n * C * NC1;
    TIO* __restrict__ oe = out + n * C * NCO;
    for (int64_t m = tid >> 6; m < tiles; m += kPreThreads / 64) {
        const int64_t c = 16 * m + col;
        const bool cv = c < C;
        float b[KS][4];
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int k1 = 16 * s + 4 * g + j;
                const bool ok = cv && k1 < NC1 && !(blk1 > 0 && (k1 == 0 || k1 == 2 * blk1));
                b[s][j] = ok ? to_f32(xe[c * NC1 + k1]) : 0.f;
            }
        v4f acc[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            acc[t] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const v4f a = *reinterpret_cast<const v4f*>(&Kt[(16 * t + col) * KST + 16 * s + 4 * g]);
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[s][j], acc[t], 0, 0, 0);
            }
        }
        if (cv) {
            TIO* __restrict__ dst = oe + c * NCO;
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int k3 = 16 * t + 4 * g + i;
                    if (k3 < NCO) dst[k3] = from_f32<TIO>(acc[t][i]);
                }
        }
    }
}

template <typename TIO, int KS, int NT>
hipError_t launch_pre(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float*,
                      const uint32_t* aux, hipStream_t stream) {
    if (aux == nullptr || cpx2 <= 0 || units % cpx2 != 0) return hipErrorInvalidValue;
    const int64_t edges = units / cpx2;
    if (edges > 0x7fffffff) return hipErrorInvalidValue;
    if (edges == 0) return hipSuccess;
    hipLaunchKernelGGL((spingtp_fwd_pre_kernel<TIO, KS, NT>), dim3(static_cast<unsigned>(edges)), dim3(kPreThreads), 0,
                       stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2), static_cast<TIO*>(out), cpx2,
                       aux);
    return hipGetLastError();
}

template <int KS, int NT>
constexpr int pre_lds_bytes() {
    return (16 * NT * (16 * KS + 4) + kPreMaxNC) * 4;
}

#define SPINGTP_PRE_ROW(KS)                                                                      \
    {{KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 1>(), 5, &launch_pre<float, KS, 1>},     \
      KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 1>(), 5, &launch_pre<uint16_t, KS, 1>}}, \
     {KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 2>(), 5, &launch_pre<float, KS, 2>},     \
      KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 2>(), 5, &launch_pre<uint16_t, KS, 2>}}, \
     {KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 3>(), 5, &launch_pre<float, KS, 3>},     \
      KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 3>(), 5, &launch_pre<uint16_t, KS, 3>}}, \
     {KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 4>(), 5, &launch_pre<float, KS, 4>},     \
      KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 4>(), 5, &launch_pre<uint16_t, KS, 4>}}, \
     {KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 5>(), 5, &launch_pre<float, KS, 5>},     \
      KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, 5>(), 5, &launch_pre<uint16_t, KS, 5>}}}

// [KS - 1][NT - 1][dtype]
const KernelEntry kPre[5][5][2] = {SPINGTP_PRE_ROW(1), SPINGTP_PRE_ROW(2), SPINGTP_PRE_ROW(3), SPINGTP_PRE_ROW(4),
                                   SPINGTP_PRE_ROW(5)};
#undef SPINGTP_PRE_ROW

}  // namespace

const KernelEntry* find_pre_kernel(int L1, int L2, int LO, int spin_mode, int dtype) {
    const int ns = spin_mode ? 3 : 1;
    const int nc1 = ns * (L1 + 1) * (L1 + 1), nc2 = ns * (L2 + 1) * (L2 + 1), nco = ns * (LO + 1) * (LO + 1);
    if (nc1 > kPreMaxNC || nc2 > kPreMaxNC || nco > kPreMaxNC || dtype < 0 || dtype > 1) return nullptr;
    return &kPre[(nc1 + 15) / 16 - 1][(nco + 15) / 16 - 1][dtype];
}

}  // namespace spingtp
