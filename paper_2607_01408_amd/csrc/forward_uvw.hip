// Fully connected SpinGTP product (mode uvw of App. E.1; Sec. 3.5 eq. spin_gtp) on gfx950.
//
// For every path p = (rho1, rho2 -> rho3) the product forms
//   R_p[n, (u, v), m3] = sum over the entries (k1, k2, m3) of p of T x1[n, u, k1] x2[n, v, k2]
// and mixes the channels:
//   out[n, w, o3 + m3] = sum_p sum_(u, v) W[p, u, v, w] R_p[n, (u, v), m3],
// o3 the first slot of rho3.  Per path and over all edges the mixing is a dense product
// [W x UV] . [UV x (edges x d3)], so it runs on the matrix cores with fp32 operands and
// sums (v_mfma_f32_32x32x2_f32): output channels w are the M dimension, the (u, v) pairs
// the K dimension and the 32 edges of a tile the N dimension, with one accumulator per
// output component m3.
//
// Mapping.  A workgroup owns 32 edges, one output block rho3, 128 output channels and
// up to 8 of the block's components; wave i owns channels 32 i .. 32 i + 31 of the 128.
// For every path into the block and every 32 (u, v) pairs:
//   (1) the 256 threads form R for 32 pairs x 32 edges x 8 components into LDS, laid out
//       [pair][component][edge] (a lane's B operand is one conflict-free LDS read);
//   (2) each wave multiplies: A = W[p, pair, w] from global memory (lanes 0..31 read 32
//       consecutive channels), B = R from LDS, 16 K steps of two pairs per component.
// The accumulators stay in registers across the paths of the block; the tile is written
// once at the end.  Blocks reached by no path and slots with l < |s| hold no entry: a
// fill kernel writes the whole output 0 first, in the same stream.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace spingtp {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f_ __attribute__((ext_vector_type(4)));

constexpr int kEdges = 32;    // N of the matrix-core product: edges of a tile
constexpr int kPairs = 32;    // (u, v) pairs staged per round (16 K steps of two)
constexpr int kGroupW = 128;  // output channels of a workgroup (4 waves x 32)
constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void spingtp_fill_zero_kernel(float* __restrict__ out, int64_t n) {
    const int64_t n4 = n >> 2;
    v4f_* o4 = reinterpret_cast<v4f_*>(out);
    const v4f_ z = {0.f, 0.f, 0.f, 0.f};
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n4;
         i += static_cast<int64_t>(gridDim.x) * kThreads)
        o4[i] = z;
    const int64_t t = 4 * n4 + static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (t < n) out[t] = 0.f;
}

__global__ __launch_bounds__(kThreads) void spingtp_fwd_uvw_kernel(const float* __restrict__ x1,
                                                                   const float* __restrict__ x2,
                                                                   const float* __restrict__ wt,
                                                                   float* __restrict__ out, int64_t N, int U, int V,
                                                                   int W, const uint32_t* __restrict__ tab,
                                                                   int n_chunks, int nco) {
    __shared__ float R[kPairs * kUvwChunk * kEdges];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kEdges;
    const uint32_t* blk = tab + kUvwHeader + 4 * blockIdx.y;
    const int o3 = static_cast<int>(blk[0]), d3 = static_cast<int>(blk[1]);
    const int rec_first = static_cast<int>(blk[2]), n_rec = static_cast<int>(blk[3]);
    const int wg = static_cast<int>(blockIdx.z) / n_chunks;
    const int m0 = (static_cast<int>(blockIdx.z) - wg * n_chunks) * kUvwChunk;
    if (m0 >= d3) return;  // the whole workgroup: this block has fewer components
    const int mc = d3 - m0 < kUvwChunk ? d3 - m0 : kUvwChunk;
    const int nc1 = static_cast<int>(tab[2]), nc2 = static_cast<int>(tab[3]);
    const uint32_t* recs = tab + tab[6];
    const uint32_t* ent = tab + tab[7];
    const int UV = U * V;
    const int wbase = wg * kGroupW + 32 * wave;  // this wave's first output channel
    const bool wave_on = wbase < W;
    const int w_lane = wbase + (lane & 31);
    const int half = lane >> 5;

    v16f acc[kUvwChunk];
#pragma unroll
    for (int j = 0; j < kUvwChunk; ++j) acc[j] = v16f{};

    for (int q = 0; q < n_rec; ++q) {
        const uint32_t* rec = recs + 4 * (rec_first + q);
        const uint32_t* csr = tab + rec[2] + m0;  // entry offsets of components m0 .. m0 + mc
        const float* __restrict__ wp = wt + static_cast<int64_t>(rec[0]) * UV * W;
        for (int c0 = 0; c0 < UV; c0 += kPairs) {
            // (1) R of pairs c0 .. c0 + 31 for the tile's edges, components m0 .. m0 + mc - 1
            for (int it = tid; it < kPairs * kEdges; it += kThreads) {
                const int pl = it >> 5, e = it & 31;
                const int pr = c0 + pl;
                const int64_t n = e0 + e;
                float r[kUvwChunk];
#pragma unroll
                for (int j = 0; j < kUvwChunk; ++j) r[j] = 0.f;
                if (pr < UV && n < N) {
                    const int u = pr / V, v = pr - u * V;
                    const float* __restrict__ a = x1 + (n * U + u) * nc1;
                    const float* __restrict__ b = x2 + (n * V + v) * nc2;
#pragma unroll
                    for (int j = 0; j < kUvwChunk; ++j) {
                        if (j < mc) {
                            float s = 0.f;
                            for (uint32_t k = csr[j]; k < csr[j + 1]; ++k) {
                                const uint32_t ix = ent[2 * k];
                                s = fmaf(__uint_as_float(ent[2 * k + 1]) * a[ix & 0xffffu], b[ix >> 16], s);
                            }
                            r[j] = s;
                        }
                    }
                }
#pragma unroll
                for (int j = 0; j < kUvwChunk; ++j) R[(pl * kUvwChunk + j) * kEdges + e] = r[j];
            }
            __syncthreads();
            // (2) out[w, edge] += W[p, pair, w] R[pair, edge] for each component
            if (wave_on) {
#pragma unroll 2
                for (int kk = 0; kk < kPairs; kk += 2) {
                    const int pr = c0 + kk + half;
                    const float av = (pr < UV && w_lane < W) ? wp[static_cast<int64_t>(pr) * W + w_lane] : 0.f;
                    const float* rb = R + ((kk + half) * kUvwChunk) * kEdges + (lane & 31);
#pragma unroll
                    for (int j = 0; j < kUvwChunk; ++j)
                        if (j < mc) acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, rb[j * kEdges], acc[j], 0, 0, 0);
                }
            }
            __syncthreads();
        }
    }

    // (3) accumulator element i of lane l holds channel wbase + 8 (i / 4) + 4 (l / 32) + i % 4
    //     and edge e0 + l % 32
    if (!wave_on) return;
    const int64_t n = e0 + (lane & 31);
    if (n >= N) return;
#pragma unroll
    for (int j = 0; j < kUvwChunk; ++j) {
        if (j >= mc) break;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int w = wbase + 8 * (i >> 2) + 4 * half + (i & 3);
            if (w < W) out[(n * W + w) * nco + o3 + m0 + j] = acc[j][i];
        }
    }
}

}  // namespace

hipError_t launch_fwd_uvw(const float* x1, const float* x2, const float* w, float* out, int64_t N, int U, int V,
                          int W, const uint32_t* table, int n_blocks, int max_d3, int nco, hipStream_t stream) {
    const int64_t total = N * W * nco;
    if (total > 0) {
        const int64_t want = (total / 4 + kThreads - 1) / kThreads;
        const unsigned g = static_cast<unsigned>(want < 4096 ? (want < 1 ? 1 : want) : 4096);
        hipLaunchKernelGGL(spingtp_fill_zero_kernel, dim3(g), dim3(kThreads), 0, stream, out, total);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (N == 0 || U == 0 || V == 0 || W == 0 || n_blocks == 0) return hipSuccess;
    const int64_t gx = (N + kEdges - 1) / kEdges;
    const int n_chunks = (max_d3 + kUvwChunk - 1) / kUvwChunk;
    const int64_t gz = static_cast<int64_t>((W + kGroupW - 1) / kGroupW) * n_chunks;
    if (gx > 0x7fffffff || n_blocks > 65535 || gz > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(spingtp_fwd_uvw_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(n_blocks),
                                                     static_cast<unsigned>(gz)),
                       dim3(kThreads), 0, stream, x1, x2, w, out, N, U, V, W, table, n_chunks, nco);
    return hipGetLastError();
}

}  // namespace spingtp

extern "C" spingtp_status spingtp_forward_fully_connected(spingtp_plan plan, const void* x1, const void* x2,
                                                          const float* weights, void* out, int64_t N, int64_t U,
                                                          int64_t V, int64_t W, void* stream) {
    if (plan == nullptr || N < 0 || U < 0 || V < 0 || W < 0) return SPINGTP_ERR_INVALID_ARG;
    if (plan->d_uvw == nullptr || plan->dtype != SPINGTP_FP32) return SPINGTP_ERR_UNSUPPORTED;
    if (U > 65536 || V > 65536 || W > 65536 || U * V > (int64_t{1} << 24)) return SPINGTP_ERR_INVALID_ARG;
    const int64_t nco = static_cast<int64_t>(plan->n_spins) * (plan->LO + 1) * (plan->LO + 1);
    if (N == 0 || W == 0) return SPINGTP_OK;
    if (N > (int64_t{1} << 40) / (W * nco)) return SPINGTP_ERR_INVALID_ARG;
    const auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
    if (out == nullptr || misaligned(out, 16)) return SPINGTP_ERR_INVALID_ARG;
    if (U > 0 && V > 0 && (x1 == nullptr || x2 == nullptr || weights == nullptr || misaligned(x1, 16) ||
                           misaligned(x2, 16) || misaligned(weights, 4)))
        return SPINGTP_ERR_INVALID_ARG;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SPINGTP_ERR_HIP;
    if (cur != plan->device) return SPINGTP_ERR_INVALID_ARG;
    const hipError_t e = spingtp::launch_fwd_uvw(
        static_cast<const float*>(x1), static_cast<const float*>(x2), weights, static_cast<float*>(out), N,
        static_cast<int>(U), static_cast<int>(V), static_cast<int>(W), plan->d_uvw, plan->uvw_blocks,
        plan->uvw_max_d3, static_cast<int>(nco), static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}
