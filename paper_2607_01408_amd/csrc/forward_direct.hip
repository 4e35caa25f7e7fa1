// Direct sparse-tensor SpinGTP kernel (family 6).
//
// out[u, o] = sum_{(a, b) in list(o)} value * A[u, a] * B[u, b]: the real bilinear
// map of the operation written out on its nonzero entries (the tensor T of Sec. 3.2
// eq. generalized_gaunt through the real basis of App. C, built by the plan in
// float64).  The same kernel runs the three roles of that tensor:
//   forward   A = x1, B = x2, o = k3          (T[k1, k2, k3] with a = k1, b = k2)
//   grad x1   A = grad_out, B = x2, o = k1    (a = k3, b = k2)
//   grad x2   A = grad_out, B = x1, o = k2    (a = k3, b = k1)
// It serves the shapes the Fourier kernels do not cover: the spin set {-2..2}
// (s_max = 2), degree triples without a Fourier instantiation, and the gradients
// of non-square shapes.  Its cost is the tensor's nonzero count per unit, so it
// suits the small degrees these shapes come with.
//
// One wave per workgroup, one unit per lane, 64 units per tile.  The A and B rows
// of the tile sit in LDS at odd strides (conflict-free per-lane gathers), with a
// zero column past each row that padding entries point at.  The entry list is
// wave-uniform: its words come in through scalar loads, 8 entries per 64-byte
// batch, and every lane gathers its own A and B values.  Outputs are summed in
// registers per output slot, staged in LDS and stored row-contiguously.
//
// Table (uint32 words, built by build_direct_table):
//   [0, 8)   NCA, NCB, NCO, STA, STB, STO, NBATCH, 0
//   [8, 8 + NCO)  batches per output slot, in output order
//   then NBATCH batches of 16 words: 8 entry words a | b << 16, 8 fp32 values,
//   and one zero batch.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.h"
#include "internal.h"

namespace spingtp {
namespace {

__device__ __forceinline__ float direct_load(const float* p) { return *p; }
__device__ __forceinline__ float direct_load(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ void direct_store(float* p, float v) { *p = v; }
__device__ __forceinline__ void direct_store(uint16_t* p, float v) { *p = f32_to_bf16(v); }

// Rows [row0, row0 + nvalid) of a [rows][nc] array into an LDS tile of stride st;
// row r of the tile reads source row (row0 + r) / per_row.  Columns nc..st-1 and
// rows past nvalid are zero.
template <typename TIO>
__device__ void direct_load_tile(const TIO* __restrict__ src, int64_t row0, int64_t per_row, int nvalid, int nc,
                                 int st, float* dst, int lane) {
    if (per_row == 1) {
        const TIO* s = src + row0 * nc;
        const int n = nvalid * nc;
        int r = lane / nc, c = lane - (lane / nc) * nc;
        const int dr = kDirectUnits / nc, dc = kDirectUnits - (kDirectUnits / nc) * nc;
        for (int e = lane; e < n; e += kDirectUnits) {
            dst[r * st + c] = direct_load(s + e);
            r += dr;
            c += dc;
            if (c >= nc) {
                c -= nc;
                ++r;
            }
        }
    } else {
        for (int r = 0; r < nvalid; ++r) {
            const TIO* s = src + ((row0 + r) / per_row) * nc;
            for (int c = lane; c < nc; c += kDirectUnits) dst[r * st + c] = direct_load(s + c);
        }
    }
    for (int r = 0; r < kDirectUnits; ++r)
        for (int c = (r < nvalid ? nc : 0) + lane; c < st; c += kDirectUnits) dst[r * st + c] = 0.f;
}

// LDS (dynamic, sized by the launch): A, B and output tiles of 64 rows each.
template <typename TIO>
__global__ __launch_bounds__(kDirectUnits) void spingtp_fwd_direct_kernel(const TIO* __restrict__ a,
                                                                          const TIO* __restrict__ b,
                                                                          TIO* __restrict__ out, int64_t units,
                                                                          int64_t cpb,
                                                                          const uint32_t* __restrict__ tab,
                                                                          int lds_floats) {
    extern __shared__ float lds[];
    const int nca = static_cast<int>(tab[0]), ncb = static_cast<int>(tab[1]), nco = static_cast<int>(tab[2]);
    const int sta = static_cast<int>(tab[3]), stb = static_cast<int>(tab[4]), sto = static_cast<int>(tab[5]);
    if (kDirectUnits * (sta + stb + sto) > lds_floats) return;  // the launch sizes LDS from the same table
    const int nbatch = static_cast<int>(tab[6]);
    const uint32_t* __restrict__ counts = tab + 8;
    const uint32_t* __restrict__ batches = tab + 8 + nco;
    float* A = lds;
    float* B = A + kDirectUnits * sta;
    float* Y = B + kDirectUnits * stb;
    const int lane = threadIdx.x;
    const float* Arow = A + lane * sta;
    const float* Brow = B + lane * stb;
    const int64_t tiles = (units + kDirectUnits - 1) / kDirectUnits;

    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int64_t u0 = tile * kDirectUnits;
        const int nvalid = static_cast<int>(units - u0 < kDirectUnits ? units - u0 : kDirectUnits);
        __syncthreads();  // the previous tile's output is stored
        direct_load_tile(a, u0, 1, nvalid, nca, sta, A, lane);
        direct_load_tile(b, u0, cpb, nvalid, ncb, stb, B, lane);
        __syncthreads();

        // one pass over all batches; the next batch's words load while this one runs
        // (the table ends with one zero batch, so that load stays inside it)
        int o = 0, left = static_cast<int>(counts[0]);
        float acc0 = 0.f, acc1 = 0.f;
        uint32_t cur[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) cur[i] = batches[i];
        for (int j = 0; j < nbatch; ++j) {
            while (left == 0) {  // output o is complete
                Y[lane * sto + o] = acc0 + acc1;
                acc0 = acc1 = 0.f;
                ++o;
                left = static_cast<int>(counts[o]);
            }
            uint32_t nxt[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) nxt[i] = batches[16 * (j + 1) + i];
#pragma unroll
            for (int i = 0; i < 8; i += 2) {
                const uint32_t w0 = cur[i], w1 = cur[i + 1];
                acc0 = fmaf(__uint_as_float(cur[8 + i]), Arow[w0 & 0xffffu] * Brow[w0 >> 16], acc0);
                acc1 = fmaf(__uint_as_float(cur[9 + i]), Arow[w1 & 0xffffu] * Brow[w1 >> 16], acc1);
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) cur[i] = nxt[i];
            --left;
        }
        for (; o < nco; ++o) {  // the last output with entries, then those without
            Y[lane * sto + o] = acc0 + acc1;
            acc0 = acc1 = 0.f;
        }
        __syncthreads();

        TIO* dst = out + u0 * nco;
        const int n = nvalid * nco;
        int r = lane / nco, c = lane - (lane / nco) * nco;
        const int dr = kDirectUnits / nco, dc = kDirectUnits - (kDirectUnits / nco) * nco;
        for (int e = lane; e < n; e += kDirectUnits) {
            direct_store(dst + e, Y[r * sto + c]);
            r += dr;
            c += dc;
            if (c >= nco) {
                c -= nco;
                ++r;
            }
        }
    }
}

template <typename TIO>
hipError_t launch_direct(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2,
                         const uint32_t* aux, int lds_floats, hipStream_t stream) {
    if (aux == nullptr || cpx2 <= 0 || units % cpx2 != 0 || lds_floats <= 0 || lds_floats > kDirectMaxLdsFloats)
        return hipErrorInvalidValue;
    const size_t bytes = static_cast<size_t>(lds_floats) * sizeof(float);
    if (bytes > 65536) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&spingtp_fwd_direct_kernel<TIO>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
        if (e != hipSuccess) return e;
    }
    const int64_t tiles = (units + kDirectUnits - 1) / kDirectUnits;
    const int64_t grid = tiles < (int64_t{1} << 20) ? tiles : (int64_t{1} << 20);
    hipLaunchKernelGGL((spingtp_fwd_direct_kernel<TIO>), dim3(static_cast<unsigned>(grid)), dim3(kDirectUnits),
                       bytes, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                       static_cast<TIO*>(out), units, cpx2, aux, lds_floats);
    return hipGetLastError();
}

const KernelEntry kDirect[2] = {{1, kDirectUnits, 0, 6, nullptr, nullptr, launch_direct<float>},
                                {1, kDirectUnits, 0, 6, nullptr, nullptr, launch_direct<uint16_t>}};

}  // namespace

const KernelEntry* find_direct_kernel(int lds_floats, int dtype) {
    if (dtype < 0 || dtype > 1 || lds_floats <= 0 || lds_floats > kDirectMaxLdsFloats) return nullptr;
    return &kDirect[dtype];
}

}  // namespace spingtp
