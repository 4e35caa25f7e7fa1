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
// Four waves per workgroup share one tile of 64 units (one unit per lane) and split
// its output slots into four ranges of about equal entry counts, so that a tile's
// LDS serves four waves of latency hiding.  The A and B rows of the tile sit in
// LDS at odd strides (conflict-free per-lane gathers), with a zero column past
// each row that padding entries point at.  The entry list is
// wave-uniform: it comes in through scalar loads, 16 entries per 96-byte batch,
// one batch ahead, and every lane gathers its own A and B values.  Entries take
// 6 bytes (two 8-bit indices, an fp32 value) so that the list of the small
// shapes this kernel serves stays inside the scalar cache (16 KB; 2,003 entries
// at degree 2 with spins {-2..2}); with 8-byte entries misses there set the pace.
// The bound is then the per-entry work: two LDS gathers and four VALU
// instructions (two address adds, a product, an fma).
// Outputs are summed in registers per output slot and stored by each lane to its
// own row as soon as the slot is complete (no output tile in LDS, which keeps
// more waves resident).
//
// Table (uint32 words, built by build_direct_table):
//   [0, 8)   NCA, NCB, NCO, STA, STB, STO, NBATCH, 16 (entries per batch)
//   [8, 13)  SEG: output-slot boundaries of the four waves (0 ... NCO)
//   [13, 18) BSEG: the first batch of each wave's range, then NBATCH
//   [18, 18 + NCO)  batches per output slot, in output order
//   then NBATCH batches of 24 words: 8 index words (entry 2i in the low half of
//   word i, entry 2i + 1 in the high half; each half a | b << 8), 16 fp32 values;
//   and two zero batches.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>

#include "device_common.h"
#include "internal.h"

namespace spingtp {
namespace {

__device__ __forceinline__ float direct_load(const float* p) { return *p; }
__device__ __forceinline__ float direct_load(const uint16_t* p) { return bf16_to_f32(*p); }
// Bounds-checked stores through a buffer resource: lanes whose byte offset is at or
// past the resource's size write nothing, so the store needs no divergent branch.
__device__ __forceinline__ void direct_store(__amdgpu_buffer_rsrc_t r, int idx, float v, float*) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, idx * 4, 0, 0);
}
__device__ __forceinline__ void direct_store(__amdgpu_buffer_rsrc_t r, int idx, float v, uint16_t*) {
    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(v), r, idx * 2, 0, 0);
}
// word 3 of a raw (untyped, stride 0) buffer resource: 32-bit data format
constexpr int kRawBufferWord3 = 0x00020000;

// Rows [row0, row0 + nvalid) of a [rows][nc] array into an LDS tile of stride st,
// by all kDirectThreads threads; row r of the tile reads source row
// (row0 + r) / per_row.  Columns nc..st-1 and rows past nvalid are zero.  Elements
// go in chunks of 8 per thread, all loads of a chunk issued before its LDS stores.
template <typename TIO>
__device__ void direct_load_tile(const TIO* __restrict__ src, int64_t row0, int64_t per_row, int nvalid, int nc,
                                 int st, float* dst, int tid) {
    constexpr int K = 8, T = kDirectThreads;
    const int n = nvalid * nc;
    int r = tid / nc, c = tid - (tid / nc) * nc;  // tile position of element e = tid + T i
    const int dr = T / nc, dc = T - (T / nc) * nc;
    for (int e0 = 0; e0 < n; e0 += K * T) {
        float v[K];
        int rr = r, cc = c;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const int e = e0 + tid + T * i;
            const int64_t at = per_row == 1 ? row0 * nc + e : ((row0 + rr) / per_row) * nc + cc;
            v[i] = e < n ? direct_load(src + at) : 0.f;
            rr += dr;
            cc += dc;
            if (cc >= nc) {
                cc -= nc;
                ++rr;
            }
        }
#pragma unroll
        for (int i = 0; i < K; ++i) {
            if (e0 + tid + T * i < n) dst[r * st + c] = v[i];
            r += dr;
            c += dc;
            if (c >= nc) {
                c -= nc;
                ++r;
            }
        }
    }
    for (int e = (nvalid * st) + tid; e < kDirectUnits * st; e += T) dst[e] = 0.f;  // rows past nvalid
    for (int r2 = tid; r2 < nvalid; r2 += T)
        for (int c2 = nc; c2 < st; ++c2) dst[r2 * st + c2] = 0.f;  // the zero column(s)
}

// LDS (dynamic, sized by the launch): A and B tiles of 64 rows each, shared by the
// workgroup's kDirectWaves waves; wave w owns the output slots
// [SEG[w], SEG[w + 1]) and walks their entries from batch BSEG[w].
template <typename TIO>
__global__ __launch_bounds__(kDirectThreads) void spingtp_fwd_direct_kernel(const TIO* __restrict__ a,
                                                                            const TIO* __restrict__ b,
                                                                            TIO* __restrict__ out, int64_t units,
                                                                            int64_t cpb,
                                                                            const uint32_t* __restrict__ tab,
                                                                            int lds_floats) {
    extern __shared__ float lds[];
    const int nca = static_cast<int>(tab[0]), ncb = static_cast<int>(tab[1]), nco = static_cast<int>(tab[2]);
    const int sta = static_cast<int>(tab[3]), stb = static_cast<int>(tab[4]);
    if (kDirectUnits * (sta + stb) > lds_floats) return;  // the launch sizes LDS from the same table
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t* __restrict__ seg = tab + 8;
    const int o_begin = static_cast<int>(seg[wave]), o_end = static_cast<int>(seg[wave + 1]);
    const int b_begin = static_cast<int>(seg[kDirectWaves + 1 + wave]);
    const int nbatch = static_cast<int>(seg[kDirectWaves + 2 + wave]) - b_begin;
    const uint32_t* __restrict__ counts = tab + 8 + 2 * (kDirectWaves + 1);
    const uint32_t* __restrict__ batches = counts + nco + 24 * b_begin;
    float* A = lds;
    float* B = A + kDirectUnits * sta;
    const float* Arow = A + lane * sta;
    const float* Brow = B + lane * stb;
    const int64_t tiles = (units + kDirectUnits - 1) / kDirectUnits;

    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int64_t u0 = tile * kDirectUnits;
        const int nvalid = static_cast<int>(units - u0 < kDirectUnits ? units - u0 : kDirectUnits);
        __syncthreads();  // every wave is done with the previous tile's rows
        direct_load_tile(a, u0, 1, nvalid, nca, sta, A, tid);
        direct_load_tile(b, u0, cpb, nvalid, ncb, stb, B, tid);
        __syncthreads();
        if (o_begin >= o_end) continue;

        // one pass over this wave's batches, two buffers: the next batch's words load
        // while this one runs (the table ends with two zero batches, so those loads stay
        // inside it).  Each lane stores its own output row; rows past nvalid fall outside
        // the buffer.
        const __amdgpu_buffer_rsrc_t dst = __builtin_amdgcn_make_buffer_rsrc(
            out + u0 * nco, 0, nvalid * nco * static_cast<int>(sizeof(TIO)), kRawBufferWord3);
        const int row = lane * nco;
        int o = o_begin, left = static_cast<int>(counts[o_begin]);
        float acc0 = 0.f, acc1 = 0.f;
        auto next_output = [&]() {  // output o is complete
            direct_store(dst, row + o, acc0 + acc1, out);
            acc0 = acc1 = 0.f;
            ++o;
            left = static_cast<int>(counts[o]);
        };
        auto run = [&](const uint32_t* w) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                acc0 = fmaf(__uint_as_float(w[8 + 2 * i]), Arow[w[i] & 0xffu] * Brow[(w[i] >> 8) & 0xffu], acc0);
                acc1 = fmaf(__uint_as_float(w[9 + 2 * i]), Arow[(w[i] >> 16) & 0xffu] * Brow[w[i] >> 24], acc1);
            }
        };
        uint32_t b0[24], b1[24];
#pragma unroll
        for (int i = 0; i < 24; ++i) b0[i] = batches[i];
        for (int j = 0; j < nbatch; j += 2) {
#pragma unroll
            for (int i = 0; i < 24; ++i) b1[i] = batches[24 * (j + 1) + i];
            while (left == 0) next_output();
            run(b0);
            --left;
            if (j + 1 >= nbatch) break;
#pragma unroll
            for (int i = 0; i < 24; ++i) b0[i] = batches[24 * (j + 2) + i];
            while (left == 0) next_output();
            run(b1);
            --left;
        }
        direct_store(dst, row + o, acc0 + acc1, out);  // the last slot with entries
        for (++o; o < o_end; ++o) direct_store(dst, row + o, 0.f, out);  // then those without
    }
}

template <typename TIO>
hipError_t launch_direct(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2,
                         const uint32_t* aux, int lds_floats, hipStream_t stream) {
    if (aux == nullptr || cpx2 <= 0 || units % cpx2 != 0 || lds_floats <= 0 || lds_floats > kDirectMaxLdsFloats)
        return hipErrorInvalidValue;
    const size_t bytes = static_cast<size_t>(lds_floats) * sizeof(float);
    if (bytes > 65536) {  // raise the dynamic LDS limit once per device (to the kernel's maximum)
        constexpr int kMaxDevices = 64;
        static std::atomic<bool> raised[kMaxDevices];
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
        if (!raised[dev].load(std::memory_order_acquire)) {
            const hipError_t e =
                hipFuncSetAttribute(reinterpret_cast<const void*>(&spingtp_fwd_direct_kernel<TIO>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                    static_cast<int>(kDirectMaxLdsFloats * sizeof(float)));
            if (e != hipSuccess) return e;
            raised[dev].store(true, std::memory_order_release);
        }
    }
    const int64_t tiles = (units + kDirectUnits - 1) / kDirectUnits;
    const int64_t grid = tiles < (int64_t{1} << 20) ? tiles : (int64_t{1} << 20);
    hipLaunchKernelGGL((spingtp_fwd_direct_kernel<TIO>), dim3(static_cast<unsigned>(grid)), dim3(kDirectThreads),
                       bytes, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                       static_cast<TIO*>(out), units, cpx2, aux, lds_floats);
    return hipGetLastError();
}

const KernelEntry kDirect[2] = {{kDirectWaves, kDirectUnits, 0, 6, nullptr, nullptr, launch_direct<float>},
                                {kDirectWaves, kDirectUnits, 0, 6, nullptr, nullptr, launch_direct<uint16_t>}};

}  // namespace

const KernelEntry* find_direct_kernel(int lds_floats, int dtype) {
    if (dtype < 0 || dtype > 1 || lds_floats <= 0 || lds_floats > kDirectMaxLdsFloats) return nullptr;
    return &kDirect[dtype];
}

}  // namespace spingtp
