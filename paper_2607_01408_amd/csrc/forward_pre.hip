// Precontracted SpinGTP for an edge input shared by the channels of an edge
// (edge multiplicity V = 1; paper Sec. 3.4, the precontraction equations, and
// App. E, depthwise mode with V = 1 and unit weights).
//
// With x2 the same for every channel c of edge n, the bilinear map
//   out[n,c,k3] = sum_{k1,k2} T[k1,k2,k3] x1[n,c,k1] x2[n,k2]
// factors into an edge kernel K_n[k1,k3] = sum_{k2} T[k1,k2,k3] x2[n,k2] (built
// once per edge) and a dense product out[n,c,:] = x1[n,c,:] K_n over the
// channels.  T is the real tensor of the operation (Sec. 3.2 eq. generalized_gaunt
// through the real basis of App. C), built on the host in float64 by the plan
// and stored as a sparse list per output entry (k1, k3).
//
// One workgroup per edge: x2 row -> LDS; K_n -> LDS (one thread per entry, a
// short gather over its k2 list, no atomics); then the channels in chunks of 64:
// x1 rows -> LDS (coalesced), each thread forms outputs (c, k3) as an fp32 dot
// product over k1 and stores them coalesced along the output row.  The l = 0
// slots of the |s| = 1 sectors are not data: they are zeroed on load, and the
// kernel's columns for them are zero, so those outputs are written as 0.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.h"
#include "internal.h"

namespace spingtp {
namespace {

constexpr int kPreThreads = 256;
constexpr int kPreChunk = 64;  // channels per x1 chunk

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

// aux words: NC1, NC2, NCO, nnz, BLK1 (0 for spins {0}), then rows[NC1 NCO + 1],
// k2[nnz] (int32) and val[nnz] (fp32 bits).
template <typename TIO>
__global__ __launch_bounds__(kPreThreads) void spingtp_fwd_pre_kernel(const TIO* __restrict__ x1,
                                                                      const TIO* __restrict__ x2,
                                                                      TIO* __restrict__ out, int64_t C,
                                                                      const uint32_t* __restrict__ aux) {
    const int NC1 = static_cast<int>(aux[0]), NC2 = static_cast<int>(aux[1]), NCO = static_cast<int>(aux[2]);
    const int nnz = static_cast<int>(aux[3]), blk1 = static_cast<int>(aux[4]);
    const int* __restrict__ rows = reinterpret_cast<const int*>(aux + 5);
    const int* __restrict__ k2s = rows + NC1 * NCO + 1;
    const float* __restrict__ vals = reinterpret_cast<const float*>(k2s + nnz);

    __shared__ float K[kPreMaxNC * kPreMaxNC];
    __shared__ float X2[kPreMaxNC];
    __shared__ float X1[kPreChunk * kPreMaxNC];

    const int tid = threadIdx.x;
    const int64_t n = blockIdx.x;
    for (int i = tid; i < NC2; i += kPreThreads) X2[i] = to_f32(x2[n * NC2 + i]);
    __syncthreads();
    for (int e = tid; e < NC1 * NCO; e += kPreThreads) {
        float acc = 0.f;
        for (int i = rows[e]; i < rows[e + 1]; ++i) acc = fmaf(vals[i], X2[k2s[i]], acc);
        K[e] = acc;
    }
    for (int64_t c0 = 0; c0 < C; c0 += kPreChunk) {
        const int cb = static_cast<int>(C - c0 < kPreChunk ? C - c0 : kPreChunk);
        const TIO* __restrict__ src = x1 + (n * C + c0) * NC1;
        __syncthreads();  // K complete; the previous chunk's X1 no longer read
        for (int i = tid; i < cb * NC1; i += kPreThreads) {
            const int k = i % NC1;
            X1[i] = (blk1 > 0 && (k == 0 || k == 2 * blk1)) ? 0.f : to_f32(src[i]);
        }
        __syncthreads();
        TIO* __restrict__ dst = out + (n * C + c0) * NCO;
        for (int o = tid; o < cb * NCO; o += kPreThreads) {
            const int c = o / NCO, k3 = o - c * NCO;
            const float* __restrict__ xr = X1 + c * NC1;
            float acc = 0.f;
            for (int k1 = 0; k1 < NC1; ++k1) acc = fmaf(xr[k1], K[k1 * NCO + k3], acc);
            dst[o] = from_f32<TIO>(acc);
        }
    }
}

template <typename TIO>
hipError_t launch_pre(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float*,
                      const uint32_t* aux, hipStream_t stream) {
    if (aux == nullptr || cpx2 <= 0 || units % cpx2 != 0) return hipErrorInvalidValue;
    const int64_t edges = units / cpx2;
    if (edges > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((spingtp_fwd_pre_kernel<TIO>), dim3(static_cast<unsigned>(edges)), dim3(kPreThreads), 0, stream,
                       static_cast<const TIO*>(x1), static_cast<const TIO*>(x2), static_cast<TIO*>(out), cpx2, aux);
    return hipGetLastError();
}

const KernelEntry kPreFp32{kPreThreads / 64, 1, static_cast<int>((kPreMaxNC * kPreMaxNC + kPreMaxNC + kPreChunk * kPreMaxNC) * 4),
                           5, &launch_pre<float>};
const KernelEntry kPreBf16{kPreThreads / 64, 1, static_cast<int>((kPreMaxNC * kPreMaxNC + kPreMaxNC + kPreChunk * kPreMaxNC) * 4),
                           5, &launch_pre<uint16_t>};

}  // namespace

const KernelEntry* find_pre_kernel(int L1, int L2, int LO, int spin_mode, int dtype) {
    const int ns = spin_mode ? 3 : 1;
    const int nc1 = ns * (L1 + 1) * (L1 + 1), nc2 = ns * (L2 + 1) * (L2 + 1), nco = ns * (LO + 1) * (LO + 1);
    if (nc1 > kPreMaxNC || nc2 > kPreMaxNC || nco > kPreMaxNC) return nullptr;
    return dtype == 0 ? &kPreFp32 : &kPreBf16;
}

}  // namespace spingtp
