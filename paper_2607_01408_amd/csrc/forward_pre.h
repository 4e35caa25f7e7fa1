// Precontracted SpinGTP kernel template (family 5) for an edge input shared by the
// channels of an edge; instantiated in forward_pre.hip (KS, NT <= 5) and
// forward_pre_large.hip (KS or NT in {7, 10}).
//
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
// Workgroups of 256 threads, each taking one edge at a time.
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
// The slots with l < |s| are not data: x1 values there are never read (taken as
// 0), and T has no entries for them, so those outputs are written as 0 and x2
// values there are never used.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
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

// Orders a wave's LDS accesses across its lanes (LDS executes a wave's
// instructions in order; this keeps the compiler from moving them).
__device__ __forceinline__ void wave_lds_order() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// Bit 4 s + j is set when x1 slot k1 = 16 s + 4 g + j (MFMA step (s, j) of lane
// group g) is data: k1 < nc1 and, in its spin block of blk1 slots (spins -S..S in
// order, so |s| = |b - ns / 2| for block b), degree l >= |s|, i.e. in-block index
// l^2 + l + m >= s^2.
template <int KS>
__device__ __forceinline__ uint64_t x1_data_mask(int nc1, int blk1, int ns, int g) {
    uint64_t m = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k1 = 16 * s + 4 * g + j;
            const int b = k1 / blk1, r = k1 - b * blk1, sa = b > ns / 2 ? b - ns / 2 : ns / 2 - b;
            if (k1 < nc1 && r >= sa * sa) m |= uint64_t{1} << (4 * s + j);
        }
    return m;
}

// KS = ceil(NC1 / 16) contraction blocks, NT = ceil(NCO / 16) output strips.
// Workgroups are persistent: workgroup b takes edges b, b + grid, ...; while an
// edge's product runs, the next edge's x2 row and each wave's first x1 tile of
// the next edge are already loading.
// WGT: per-channel path weights (spingtp_forward_v1_weighted).  The contraction
// index then runs over path slots q = (path p, x1 slot k1), the edge kernel's
// entry (q, k3) holds path p's share, and the operand of channel c at q is
// wts[c][p] x1[c][k1] (slot list in LDS), so each path is weighted per channel.
template <typename TIO, int KS, int NT, bool WGT = false>
__global__ __launch_bounds__(kPreThreads) void spingtp_fwd_pre_kernel(const TIO* __restrict__ x1,
                                                                      const TIO* __restrict__ x2,
                                                                      TIO* __restrict__ out, int64_t C,
                                                                      int64_t edges,
                                                                      const uint32_t* __restrict__ aux,
                                                                      const float* __restrict__ wts) {
    constexpr int KST = 16 * KS + 4;
    constexpr int KT_FLOATS = 16 * NT * KST;
    // row stride of a wave's staging tile (x1 rows, then output rows); the weighted
    // kernel's contraction is longer than an x1 row (at most kPreMaxNC slots)
    constexpr int RS = WGT ? (16 * NT > kPreMaxNC + 1 ? 16 * NT : kPreMaxNC + 1) + 4 : 16 * (KS > NT ? KS : NT) + 4;
    constexpr int NW = kPreThreads / 64;
    // x1 values per lane of a 16-channel tile: 16 NC1 / 64 <= 4 KS (weighted: NC1 <= 160)
    constexpr int PF = WGT ? 40 : 4 * KS;
    constexpr int PO = 4 * NT;  // output values per lane of a tile
    __shared__ __align__(16) float Kt[KT_FLOATS];
    __shared__ __align__(16) float Stage[NW * 16 * RS];
    __shared__ float X2[kPreMaxNC];
    __shared__ uint32_t QM[WGT ? 16 * KS : 1];  // path slots: x1 slot | path << 16

    // NCOL: contraction length; NC1: x1 row length (the same without weights)
    const int NCOL = static_cast<int>(aux[0]), NC2 = static_cast<int>(aux[1]), NCO = static_cast<int>(aux[2]);
    const int NC1 = WGT ? static_cast<int>(aux[12]) : NCOL;
    const int blk1 = static_cast<int>(aux[3]), ipt = static_cast<int>(aux[6]), ns = static_cast<int>(aux[11]);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, col = lane & 15, g = lane >> 4;
    // (64 mask bits hold KS <= 16; the weighted kernel compares q with NCOL instead)
    const uint64_t vmask = WGT ? 0 : x1_data_mask<(KS <= 16 ? KS : 16)>(NCOL, blk1, ns, g);
    const int npaths = WGT ? static_cast<int>(aux[13]) : 0;
    if constexpr (WGT) {
        const uint32_t* __restrict__ qs = aux + aux[14];
        for (int i = tid; i < 16 * KS; i += kPreThreads) QM[i] = i < NCOL ? qs[i] : 0u;  // read after a barrier
    }
    const int64_t tiles = (C + 15) / 16;
    const int64_t stride = gridDim.x;
    float* __restrict__ st = Stage + wave * 16 * RS;
    const uint2* __restrict__ items = reinterpret_cast<const uint2*>(aux + kPreHeader) + tid;

    float pf[PF];
    auto prefetch = [&](int64_t n, int64_t m) {
        const int cnt = static_cast<int>((C - 16 * m < 16 ? C - 16 * m : 16)) * NC1;
        const TIO* __restrict__ src = x1 + (n * C + 16 * m) * NC1;
#pragma unroll
        for (int q = 0; q < PF; ++q) {
            const int e = lane + 64 * q;
            pf[q] = e < cnt ? to_f32(src[e]) : 0.f;
        }
    };
    // Per-lane position of element lane + 64 q of a tile stored row-major in rows
    // of length nc, stepped by 64 = q nc + r.
    const int q1 = 64 / NC1, r1 = 64 - q1 * NC1, qo = 64 / NCO, ro = 64 - qo * NCO;
    const int row1 = lane / NC1, k1l = lane - row1 * NC1, rowo = lane / NCO, k3l = lane - rowo * NCO;

    int64_t n = blockIdx.x;
    float x2v = (n < edges && tid < NC2) ? to_f32(x2[n * NC2 + tid]) : 0.f;
    if (n < edges && wave < tiles) prefetch(n, wave);
    for (; n < edges; n += stride) {
        const int64_t nn = n + stride;
        uint2 ia[8], ib[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) ia[j] = items[j * kPreThreads];
        for (int i = tid; i < KT_FLOATS / 4; i += kPreThreads)
            reinterpret_cast<v4f*>(Kt)[i] = v4f{0.f, 0.f, 0.f, 0.f};
        if (tid < NC2) X2[tid] = x2v;
        __syncthreads();

        // Kernel build: the next 8 items load while the current 8 are summed; the
        // 8 x2 reads of a group are issued before its sums.
        {
            float acc = 0.f;
            auto consume = [&](const uint2 (&it)[8]) {
                float xv[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) xv[j] = X2[(it[j].x >> 16) & 0xffu];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    acc = fmaf(__uint_as_float(it[j].y), xv[j], acc);
                    if (it[j].x >> 24) {
                        Kt[it[j].x & 0xffffu] = acc;
                        acc = 0.f;
                    }
                }
            };
            for (int i = 0; i < ipt; i += 16) {  // ipt is a multiple of 8
                const bool second = i + 8 < ipt;
                if (second)
#pragma unroll
                    for (int j = 0; j < 8; ++j) ib[j] = items[(i + 8 + j) * kPreThreads];
                consume(ia);
                if (i + 16 < ipt)
#pragma unroll
                    for (int j = 0; j < 8; ++j) ia[j] = items[(i + 16 + j) * kPreThreads];
                if (second) consume(ib);
            }
        }
        if (nn < edges && tid < NC2) x2v = to_f32(x2[nn * NC2 + tid]);
        __syncthreads();

        TIO* __restrict__ oe = out + n * C * NCO;
        for (int64_t m = wave; m < tiles; m += NW) {
            const int rows = static_cast<int>(C - 16 * m < 16 ? C - 16 * m : 16);
            {  // x1 tile -> staging rows
                int r = row1, k = k1l;
#pragma unroll
                for (int q = 0; q < PF; ++q) {
                    if (lane + 64 * q < rows * NC1) st[r * RS + k] = pf[q];
                    r += q1;
                    k += r1;
                    if (k >= NC1) {
                        k -= NC1;
                        ++r;
                    }
                }
            }
            wave_lds_order();
            v4f acc[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};
            if constexpr (WGT) {
                // operands formed block by block from the staged x1 rows: channel c's value
                // at path slot q is wts[c][path] x1[c][slot]; the staged rows stay untouched
                // until the output staging below
                if (m + NW < tiles)
                    prefetch(n, m + NW);
                else if (nn < edges)
                    prefetch(nn, wave);
                const int64_t ch = 16 * m + col;  // this lane's channel of the edge
                const float* __restrict__ wc = wts + (ch < C ? ch : 0) * npaths;
#pragma unroll 2
                for (int s = 0; s < KS; ++s) {
                    float bs[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const uint32_t e = QM[16 * s + 4 * g + j];  // 0 past the slots: in-bounds reads
                        const bool use = 16 * s + 4 * g + j < NCOL && ch < C;
                        bs[j] = use ? st[col * RS + (e & 0xffffu)] * wc[e >> 16] : 0.f;
                    }
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const v4f a = *reinterpret_cast<const v4f*>(&Kt[(16 * t + col) * KST + 16 * s + 4 * g]);
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], bs[j], acc[t], 0, 0, 0);
                    }
                }
            } else {
                float b[KS][4];
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    const v4f v = *reinterpret_cast<const v4f*>(&st[col * RS + 16 * s + 4 * g]);
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        b[s][j] = ((vmask >> (4 * s + j)) & 1u) ? v[j] : 0.f;
                    }
                }
                if (m + NW < tiles)
                    prefetch(n, m + NW);
                else if (nn < edges)
                    prefetch(nn, wave);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
#pragma unroll
                    for (int s = 0; s < KS; ++s) {
                        const v4f a = *reinterpret_cast<const v4f*>(&Kt[(16 * t + col) * KST + 16 * s + 4 * g]);
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[s][j], acc[t], 0, 0, 0);
                    }
                }
            }
            wave_lds_order();
            // outputs -> staging rows (lane: channel col, k3 = 16 t + 4 g + i), then
            // coalesced stores of the tile's contiguous output block
#pragma unroll
            for (int t = 0; t < NT; ++t) *reinterpret_cast<v4f*>(&st[col * RS + 16 * t + 4 * g]) = acc[t];
            wave_lds_order();
            {
                TIO* __restrict__ dst = oe + 16 * m * NCO;
                int r = rowo, k = k3l;
#pragma unroll
                for (int q = 0; q < PO; ++q) {
                    const int e = lane + 64 * q;
                    if (e < rows * NCO) dst[e] = from_f32<TIO>(st[r * RS + k]);
                    r += qo;
                    k += ro;
                    if (k >= NCO) {
                        k -= NCO;
                        ++r;
                    }
                }
            }
            wave_lds_order();
        }
        __syncthreads();  // Kt and X2 are rewritten for the next edge
    }
}

// Blocked variant for KS or NT above 5 (rows longer than 80: degree 5 or 6 with
// spins {-1, 0, +1}).  The whole transposed kernel would not leave room for two
// workgroups per CU, so its k3 rows are built and used in blocks of
// kPreBlockRows (48): per edge and per group of 128 channels, each wave first
// loads the operands of its two 16-channel tiles into registers (through its
// LDS tile), then for every block the workgroup builds the block in LDS from
// that block's items and each wave multiplies its tiles with it and writes the
// block's output columns (coalesced along the rows' 48-value segments).  Two
// resident workgroups per CU keep the matrix cores of one busy while the other
// builds.  Channels beyond 128 per edge take further groups and rebuild the
// blocks.
template <typename TIO, int KS, int NT>
__global__ __launch_bounds__(kPreThreads, 2) void spingtp_fwd_pre_blocked_kernel(const TIO* __restrict__ x1,
                                                                                 const TIO* __restrict__ x2,
                                                                                 TIO* __restrict__ out, int64_t C,
                                                                                 int64_t edges,
                                                                                 const uint32_t* __restrict__ aux) {
    constexpr int KST = 16 * KS + 4;
    constexpr int RB = kPreBlockRows;
    constexpr int SB = RB / 16;  // strips per block
    constexpr int NB3 = (16 * NT + RB - 1) / RB;
    constexpr int RS = 16 * KS + 4;  // x1 tile row stride
    constexpr int RSO = RB + 4;      // output tile row stride
    constexpr int STG = 16 * (RS > RSO ? RS : RSO);
    constexpr int NW = kPreThreads / 64;
    constexpr int TPW = 2;  // tiles per wave per channel group
    constexpr int PF = 4 * KS;
    constexpr int PO = RB / 4;  // output values per lane of a tile block
    __shared__ __align__(16) float Kb[RB * KST + kPreThreads];  // + one spare slot per thread
    __shared__ __align__(16) float Stage[NW * STG];
    __shared__ float X2[kPreMaxNC];

    const int NC1 = static_cast<int>(aux[0]), NC2 = static_cast<int>(aux[1]), NCO = static_cast<int>(aux[2]);
    const int blk1 = static_cast<int>(aux[3]), ipt = static_cast<int>(aux[6]), stride = static_cast<int>(aux[10]);
    const int ns = static_cast<int>(aux[11]);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, col = lane & 15, g = lane >> 4;
    const uint64_t vmask = x1_data_mask<KS>(NC1, blk1, ns, g);
    const int64_t tiles = (C + 15) / 16;
    float* __restrict__ st = Stage + wave * STG;
    const uint2* __restrict__ items0 = reinterpret_cast<const uint2*>(aux + kPreHeader) + tid;
    const int q1 = 64 / NC1, r1 = 64 - q1 * NC1;
    const int row1 = lane / NC1, k1l = lane - row1 * NC1;

    for (int64_t n = blockIdx.x; n < edges; n += gridDim.x) {
        const TIO* __restrict__ xe = x1 + n * C * NC1;
        TIO* __restrict__ oe = out + n * C * NCO;
        for (int64_t g0 = 0; g0 < tiles; g0 += NW * TPW) {
            // operands of this wave's tiles, through its LDS tile
            float b[TPW][KS][4];
#pragma unroll
            for (int i = 0; i < TPW; ++i) {
                const int64_t m = g0 + wave + NW * i;
                if (m < tiles) {
                    const int rows = static_cast<int>(C - 16 * m < 16 ? C - 16 * m : 16);
                    const TIO* __restrict__ src = xe + 16 * m * NC1;
                    float pf[PF];
#pragma unroll
                    for (int q = 0; q < PF; ++q) {
                        const int e = lane + 64 * q;
                        pf[q] = e < rows * NC1 ? to_f32(src[e]) : 0.f;
                    }
                    int r = row1, k = k1l;
#pragma unroll
                    for (int q = 0; q < PF; ++q) {
                        if (lane + 64 * q < rows * NC1) st[r * RS + k] = pf[q];
                        r += q1;
                        k += r1;
                        if (k >= NC1) {
                            k -= NC1;
                            ++r;
                        }
                    }
                    wave_lds_order();
#pragma unroll
                    for (int s = 0; s < KS; ++s) {
                        const v4f v = *reinterpret_cast<const v4f*>(&st[col * RS + 16 * s + 4 * g]);
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            b[i][s][j] = ((vmask >> (4 * s + j)) & 1u) ? v[j] : 0.f;
                        }
                    }
                    wave_lds_order();
                } else {
#pragma unroll
                    for (int s = 0; s < KS; ++s)
#pragma unroll
                        for (int j = 0; j < 4; ++j) b[i][s][j] = 0.f;
                }
            }
            for (int blk = 0; blk < NB3; ++blk) {
                __syncthreads();  // the previous block (or edge) is no longer read
                for (int i = tid; i < RB * KST / 4; i += kPreThreads)
                    reinterpret_cast<v4f*>(Kb)[i] = v4f{0.f, 0.f, 0.f, 0.f};
                if (blk == 0 && g0 == 0 && tid < NC2) X2[tid] = to_f32(x2[n * NC2 + tid]);
                __syncthreads();
                {  // build block blk
                    const uint2* __restrict__ items = items0 + static_cast<int64_t>(blk) * stride * kPreThreads;
                    float acc = 0.f;
                    uint2 ia[8], ib[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) ia[j] = items[j * kPreThreads];
                    auto consume = [&](const uint2 (&it)[8]) {
                        float xv[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j) xv[j] = X2[(it[j].x >> 16) & 0xffu];
#pragma unroll
                        for (int j = 0; j < 8; ++j) {
                            acc = fmaf(__uint_as_float(it[j].y), xv[j], acc);
                            const bool last = (it[j].x >> 24) != 0;
                            Kb[last ? static_cast<int>(it[j].x & 0xffffu) : RB * KST + tid] = acc;
                            acc = last ? 0.f : acc;
                        }
                    };
                    // ipt is a multiple of 16 and 16 zero items follow each block: every
                    // load is unconditional and runs 8 items ahead of the sums, and the
                    // stores are branch-free (a list's last item stores the sum, the
                    // others write this thread's spare slot)
                    for (int i = 0; i < ipt; i += 16) {
#pragma unroll
                        for (int j = 0; j < 8; ++j) ib[j] = items[(i + 8 + j) * kPreThreads];
                        consume(ia);
#pragma unroll
                        for (int j = 0; j < 8; ++j) ia[j] = items[(i + 16 + j) * kPreThreads];
                        consume(ib);
                    }
                }
                __syncthreads();
                // products of this wave's tiles with block blk
                v4f acc[TPW][SB];
#pragma unroll
                for (int i = 0; i < TPW; ++i)
#pragma unroll
                    for (int t = 0; t < SB; ++t) acc[i][t] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < KS; ++s)
#pragma unroll
                    for (int t = 0; t < SB; ++t) {
                        if (SB * blk + t >= NT) continue;
                        const v4f a = *reinterpret_cast<const v4f*>(&Kb[(16 * t + col) * KST + 16 * s + 4 * g]);
#pragma unroll
                        for (int i = 0; i < TPW; ++i)
#pragma unroll
                            for (int j = 0; j < 4; ++j)
                                acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[i][s][j], acc[i][t], 0, 0, 0);
                    }
                const int bw = NCO - RB * blk < RB ? NCO - RB * blk : RB;  // output columns of this block
                const int qo = 64 / bw, ro = 64 - qo * bw;
                const int rowo = lane / bw, kol = lane - rowo * bw;
#pragma unroll
                for (int i = 0; i < TPW; ++i) {
                    const int64_t m = g0 + wave + NW * i;
                    if (m >= tiles) continue;
                    const int rows = static_cast<int>(C - 16 * m < 16 ? C - 16 * m : 16);
#pragma unroll
                    for (int t = 0; t < SB; ++t)
                        if (SB * blk + t < NT) *reinterpret_cast<v4f*>(&st[col * RSO + 16 * t + 4 * g]) = acc[i][t];
                    wave_lds_order();
                    TIO* __restrict__ dst = oe + 16 * m * NCO + RB * blk;
                    int r = rowo, k = kol;
#pragma unroll
                    for (int q = 0; q < PO; ++q) {
                        if (lane + 64 * q < rows * bw) dst[static_cast<int64_t>(r) * NCO + k] = from_f32<TIO>(st[r * RSO + k]);
                        r += qo;
                        k += ro;
                        if (k >= bw) {
                            k -= bw;
                            ++r;
                        }
                    }
                    wave_lds_order();
                }
            }
        }
    }
}

// Resident workgroups of a kernel on the current device (cached per device and
// kernel; 0 on failure).
template <auto Kernel>
int64_t resident_groups() {
    constexpr int kMaxDevices = 64;
    static std::atomic<int64_t> cache[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
    int64_t v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, Kernel, kPreThreads, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    v = static_cast<int64_t>(per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1);
    cache[dev].store(v, std::memory_order_relaxed);
    return v;
}

template <typename TIO, int KS, int NT>
hipError_t launch_pre(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float*,
                      const uint32_t* aux, hipStream_t stream) {
    if (aux == nullptr || cpx2 <= 0 || units % cpx2 != 0) return hipErrorInvalidValue;
    const int64_t edges = units / cpx2;
    if (edges == 0) return hipSuccess;
    constexpr bool kBlocked = KS > 5 || NT > 5;
    int64_t resident = 0;
    if constexpr (kBlocked)
        resident = resident_groups<spingtp_fwd_pre_blocked_kernel<TIO, KS, NT>>();
    else
        resident = resident_groups<spingtp_fwd_pre_kernel<TIO, KS, NT>>();
    if (resident <= 0) return hipErrorInvalidValue;
    const int64_t grid = edges < resident ? edges : resident;
    if constexpr (kBlocked)
        hipLaunchKernelGGL((spingtp_fwd_pre_blocked_kernel<TIO, KS, NT>), dim3(static_cast<unsigned>(grid)),
                           dim3(kPreThreads), 0, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                           static_cast<TIO*>(out), cpx2, edges, aux);
    else
        hipLaunchKernelGGL((spingtp_fwd_pre_kernel<TIO, KS, NT>), dim3(static_cast<unsigned>(grid)), dim3(kPreThreads),
                           0, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                           static_cast<TIO*>(out), cpx2, edges, aux, nullptr);
    return hipGetLastError();
}

// The per-channel path-weighted kernel (one block of rows): `wts` carries the
// channel weights [C][NPATHS] (fp32) in place of the plan tables.
template <typename TIO, int KS, int NT>
hipError_t launch_pre_weighted(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2,
                               const float* wts, const uint32_t* aux, hipStream_t stream) {
    if (aux == nullptr || wts == nullptr || cpx2 <= 0 || units % cpx2 != 0) return hipErrorInvalidValue;
    const int64_t edges = units / cpx2;
    if (edges == 0) return hipSuccess;
    const int64_t resident = resident_groups<spingtp_fwd_pre_kernel<TIO, KS, NT, true>>();
    if (resident <= 0) return hipErrorInvalidValue;
    const int64_t grid = edges < resident ? edges : resident;
    hipLaunchKernelGGL((spingtp_fwd_pre_kernel<TIO, KS, NT, true>), dim3(static_cast<unsigned>(grid)),
                       dim3(kPreThreads), 0, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                       static_cast<TIO*>(out), cpx2, edges, aux, wts);
    return hipGetLastError();
}

template <int KS, int NT>
constexpr int pre_lds_bytes() {
    if constexpr (KS > 5 || NT > 5) {
        constexpr int RS = 16 * KS + 4, RSO = kPreBlockRows + 4;
        return (kPreBlockRows * (16 * KS + 4) + kPreThreads + (kPreThreads / 64) * 16 * (RS > RSO ? RS : RSO) +
                kPreMaxNC) * 4;
    } else {
        return (16 * NT * (16 * KS + 4) + (kPreThreads / 64) * 16 * (16 * (KS > NT ? KS : NT) + 4) + kPreMaxNC) * 4;
    }
}

// Launch entries {fp32, bf16} of one (KS, NT) instantiation.
#define SPINGTP_PRE_PAIR(KS, NT)                                                               \
    {KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, NT>(), 5, &launch_pre<float, KS, NT>}, \
     KernelEntry{kPreThreads / 64, 1, pre_lds_bytes<KS, NT>(), 5, &launch_pre<uint16_t, KS, NT>}}
// ... of the per-channel path-weighted kernel (always the one-block kernel)
#define SPINGTP_PRE_W_PAIR(KS, NT)                                                                         \
    {KernelEntry{kPreThreads / 64, 1,                                                                     \
                 (16 * NT * (16 * KS + 4) + (kPreThreads / 64) * 16 * (kPreMaxNC + 5) + kPreMaxNC + 16 * KS) * 4, \
                 5, &launch_pre_weighted<float, KS, NT>},                                                   \
     KernelEntry{kPreThreads / 64, 1,                                                                     \
                 (16 * NT * (16 * KS + 4) + (kPreThreads / 64) * 16 * (kPreMaxNC + 5) + kPreMaxNC + 16 * KS) * 4, \
                 5, &launch_pre_weighted<uint16_t, KS, NT>}}

}  // namespace
}  // namespace spingtp
