// Gradients of the per-channel path-weighted product with the edge input shared by
// the channels (spingtp_backward_v1_weighted; the forward is spingtp_forward_v1_weighted),
// and the same product with a per-unit second input, forward and gradients
// (spingtp_forward_weighted, spingtp_backward_weighted: App. E.1 mode uuu with
// per-channel path weights; there gx2 is per unit and x2 is staged as a tile).
//
// The forward is out[n,c,k3] = sum_p W[c,p] sum_{(k1,k2,k3) in p} T[k1,k2,k3] x1[n,c,k1] x2[n,k2]
// (App. E.1 mode uvu with V = 1 and one weight per channel and path of eq. spin_gtp,
// Sec. 3.4).  It is linear in each of x1, x2 and W, so for dL/dout = g
//   gx1[n,c,k1] = sum over the entries with k1 of W[c,p] T x2[n,k2] g[n,c,k3],
//   gx2[n,k2]   = sum_c sum over the entries with k2 of W[c,p] T x1[n,c,k1] g[n,c,k3],
//   gW[c,p]     = sum_n sum over the entries of p of T x1[n,c,k1] x2[n,k2] g[n,c,k3],
// three sums over the nonzeros of T in three orders (by k1, by k2, by path).
//
// A workgroup owns a 64-channel tile (one channel per lane) and a contiguous range
// of edges; its four waves work on the same edge and split each pass's keys into
// four ranges of about equal entry counts.  The tile's weight rows and its running
// gW sums stay in LDS for the whole range; per edge the x1 and g rows of the tile
// and the x2 row are staged in LDS (odd row strides, so the per-lane gathers are
// conflict-free, and a zero column past each row that the lists' padding entries
// point at).  The entry lists are wave-uniform: they come in through vector loads,
// 32 entries (one word per lane) a block with the next block loading meanwhile, and
// reach scalar registers by readlane, eight entries per step.  (Scalar loads would
// share their wait counter with the LDS gathers, so every gather would also wait
// for the prefetch.)
//   * gW: per path, each lane adds its channel's sum to its row of the LDS tile;
//     at the end of the range the tile goes to the workspace ([range][path][channel]);
//   * gx2: per k2, each lane sums its channel's terms in a register, and a
//     fixed-order wave reduction writes the tile's sum into the workspace row of the
//     channel tile ([tile][edge][k2]);
//   * gx1: per k1, each lane's sum goes into its x1 row in LDS (after a barrier: the
//     other passes read those rows), and the tile leaves in coalesced stores.
// Two small kernels add the partial sums of gx2 over the channel tiles and those of
// gW over the edge ranges, in a fixed order: the results do not depend on scheduling.
//
// Table (uint32 words, built by build_bwd_v1w_table):
//   [0, 16)  NC1, NC2, NCO, NP (paths), NNZ, then the word offsets of SEG1, SEG2,
//            SEGP (list boundaries, in entries: NC1 + 1, NC2 + 1, NP + 1 words) and of
//            LIST1, LIST2, LISTP; zeros
//   [11, 13) the word offsets of SEG3 (NCO + 1) and LIST3
//   [16, 36) the key ranges of the four waves: five boundaries per list (LIST1,
//            LIST2, LISTP, LIST3), 0 ... number of keys
//   each list entry is two words: a | b << 10 | c << 20, fp32 value;
//   LIST1 (per k1): a = path, b = k2, c = k3;  LIST2 (per k2): a = path, b = k1, c = k3;
//   LISTP (per path): a = k1, b = k2, c = k3;  LIST3 (per k3, the forward): a = path,
//   b = k1, c = k2.  Every segment is padded to a multiple
//   of eight entries with value 0 whose indices point at the zero columns, and every
//   list ends with 96 more of those (the prefetch of the last blocks reads them).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>

#include "device_common.h"
#include "internal.h"

namespace spingtp {
namespace {

constexpr int kBw1wLanes = 64;
constexpr int kBw1wThreads = 64 * kBw1wWaves;

__device__ __forceinline__ float bw_load(const float* p) { return *p; }
__device__ __forceinline__ float bw_load(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ void bw_store(float* p, float v) { *p = v; }
__device__ __forceinline__ void bw_store(uint16_t* p, float v) { *p = f32_to_bf16(v); }

// rows [0, nrows) of a contiguous [nrows][nc] block into an LDS tile of stride st
template <typename TIO>
__device__ __forceinline__ void bw_load_rows(const TIO* __restrict__ src, int nrows, int nc, int st, float* dst,
                                             int tid) {
    const int n = nrows * nc;
    for (int e = tid; e < n; e += kBw1wThreads) {
        const int r = e / nc;
        dst[r * st + (e - r * nc)] = bw_load(src + e);
    }
}

// One pass over keys [k0, k1) of a list: for every key k the sum over its segment of
// value * term(a, b, c), handed to emit(k, sum).  The entries are walked as one
// stream of 32-entry blocks (lane l holds word l of the block, the next block loads
// meanwhile), four 8-entry steps a block with static readlane positions; a key ends
// where its segment does (segments are multiples of 8, so at a step boundary), and
// keys with empty segments get 0.
template <typename F, typename E>
__device__ __forceinline__ void bw_pass(const uint32_t* __restrict__ seg, const uint32_t* __restrict__ list, int k0,
                                        int k1, int lane, F&& term, E&& emit) {
    int k = k0;
    int kend = k < k1 ? static_cast<int>(seg[k + 1]) : 0;
    const int e0 = static_cast<int>(seg[k0]), e1 = static_cast<int>(seg[k1]);
    while (k < k1 && kend == e0) {  // empty keys before the first entry
        emit(k, 0.f);
        ++k;
        kend = k < k1 ? static_cast<int>(seg[k + 1]) : 0;
    }
    const uint32_t* __restrict__ base = list + 2 * e0;
    uint32_t vcur = base[lane], vnxt = base[64 + lane];
    float acc0 = 0.f, acc1 = 0.f;
    for (int blk = e0; blk < e1; blk += 32) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = blk + 8 * j;
            if (e < e1) {
                uint32_t w[16];
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    w[i] = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(vcur), 16 * j + i));
#pragma unroll
                for (int i = 0; i < 8; i += 2) {
                    const uint32_t i0 = w[2 * i], i1 = w[2 * i + 2];
                    acc0 = fmaf(__uint_as_float(w[2 * i + 1]), term(i0 & 0x3ffu, (i0 >> 10) & 0x3ffu, i0 >> 20),
                                acc0);
                    acc1 = fmaf(__uint_as_float(w[2 * i + 3]), term(i1 & 0x3ffu, (i1 >> 10) & 0x3ffu, i1 >> 20),
                                acc1);
                }
                while (k < k1 && kend == e + 8) {  // keys ending here (then the empty ones after them)
                    emit(k, acc0 + acc1);
                    acc0 = acc1 = 0.f;
                    ++k;
                    kend = k < k1 ? static_cast<int>(seg[k + 1]) : 0;
                }
            }
        }
        vcur = vnxt;
        vnxt = base[2 * (blk - e0) + 128 + lane];
    }
}

// sum of v over the 64 lanes of the wave, in a fixed order (every lane gets it)
__device__ __forceinline__ float bw_wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kBw1wLanes);
    return v;
}

__host__ __device__ constexpr int bw_stride(int n) { return (n + 1) | 1; }  // odd, with a zero column

// Workgroups a launch aims for: as many as fit the chip at once (256 CUs, as many
// per CU as their LDS allows, at most 8): more edge ranges where the tile is small,
// and the weight rows amortised over more edges where it is large.
int bw_target_groups(int lds_floats) {
    const int per_cu = kBw1wMaxLdsFloats / (lds_floats > 0 ? lds_floats : 1);
    return 256 * (per_cu < 1 ? 1 : (per_cu > 8 ? 8 : per_cu));
}

// SHARED: x2 [N][NC2] shared by the channels of an edge (gx2 summed over the
// channels into the workspace); else x2 [N][C][NC2] per unit (gx2 per unit, staged
// in an LDS tile and stored with gx1).
template <typename TIO, bool SHARED>
__global__ __launch_bounds__(kBw1wThreads) void spingtp_bwd_v1w_kernel(
    const TIO* __restrict__ x1, const TIO* __restrict__ x2, const float* __restrict__ wts, const TIO* __restrict__ g,
    TIO* __restrict__ gx1, TIO* __restrict__ gx2, float* __restrict__ ws_x2, float* __restrict__ ws_w, int64_t N,
    int64_t C, int64_t epg, const uint32_t* __restrict__ tab, int64_t x2s, bool acc_gx1) {
    extern __shared__ float lds[];
    const int nc1 = static_cast<int>(tab[0]), nc2 = static_cast<int>(tab[1]), nco = static_cast<int>(tab[2]);
    const int np = static_cast<int>(tab[3]);
    const uint32_t* __restrict__ seg1 = tab + tab[5];
    const uint32_t* __restrict__ seg2 = tab + tab[6];
    const uint32_t* __restrict__ segp = tab + tab[7];
    const uint32_t* __restrict__ list1 = tab + tab[8];
    const uint32_t* __restrict__ list2 = tab + tab[9];
    const uint32_t* __restrict__ listp = tab + tab[10];
    const int stw = bw_stride(np), st1 = bw_stride(nc1), sto = bw_stride(nco), st2 = bw_stride(nc2);
    float* Wt = lds;                       // [64][stw] weights of the tile's channels
    float* GW = Wt + kBw1wLanes * stw;     // [64][stw] gW sums of the edge range
    float* X1 = GW + kBw1wLanes * stw;     // [64][st1] x1 rows, then the gx1 rows
    float* G = X1 + kBw1wLanes * st1;      // [64][sto] grad_out rows
    float* X2 = G + kBw1wLanes * sto;      // SHARED: [st2] the edge's x2 row; else [64][st2] x2 rows
    float* GX2 = X2 + kBw1wLanes * st2;    // [64][st2] gx2 rows (per-unit x2 only)

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t group = blockIdx.x, tile = blockIdx.y;
    const int64_t c0 = tile * kBw1wLanes;
    const int nch = static_cast<int>(C - c0 < kBw1wLanes ? C - c0 : kBw1wLanes);
    const int64_t n_begin = group * epg;
    const int64_t n_end = n_begin + epg < N ? n_begin + epg : N;
    // this wave's keys in each pass
    const uint32_t* __restrict__ kr = tab + 16;
    const int k1b = static_cast<int>(kr[wave]), k1e = static_cast<int>(kr[wave + 1]);
    const int k2b = static_cast<int>(kr[5 + wave]), k2e = static_cast<int>(kr[6 + wave]);
    const int kpb = static_cast<int>(kr[10 + wave]), kpe = static_cast<int>(kr[11 + wave]);

    // zero everything once (zero columns and the rows past nch stay zero: the per-edge
    // loads write only rows < nch and columns < nc), then the weight rows
    const int total = kBw1wLanes * (2 * stw + st1 + sto) + (SHARED ? st2 : 2 * kBw1wLanes * st2);
    for (int i = tid; i < total; i += kBw1wThreads) lds[i] = 0.f;
    __syncthreads();
    for (int e = tid; e < nch * np; e += kBw1wThreads) {
        const int r = e / np;
        Wt[r * stw + (e - r * np)] = wts[c0 * np + e];
    }
    const float* Wr = Wt + lane * stw;
    float* GWr = GW + lane * stw;
    float* X1r = X1 + lane * st1;
    const float* Gr = G + lane * sto;
    const float* X2r = SHARED ? X2 : X2 + lane * st2;
    float* GX2r = GX2 + lane * st2;

    for (int64_t n = n_begin; n < n_end; ++n) {
        __syncthreads();  // the previous edge's gradient rows have left
        const int64_t row0 = n * C + c0;
        bw_load_rows(x1 + row0 * nc1, nch, nc1, st1, X1, tid);
        bw_load_rows(g + row0 * nco, nch, nco, sto, G, tid);
        if constexpr (SHARED) {
            for (int k = tid; k < nc2; k += kBw1wThreads) X2[k] = bw_load(x2 + n * x2s + k);
        } else {
            bw_load_rows(x2 + row0 * nc2, nch, nc2, st2, X2, tid);
        }
        __syncthreads();

        // gW: every (channel, path) sum belongs to one wave
        bw_pass(segp, listp, kpb, kpe, lane,
                [&](uint32_t a, uint32_t b, uint32_t cc) { return X2r[b] * (X1r[a] * Gr[cc]); },
                [&](int p, float acc) { GWr[p] += acc; });
        // gx2: per k2 the sum over the tile's channels (a fixed-order wave reduction), or
        // per unit into the gx2 rows
        bw_pass(seg2, list2, k2b, k2e, lane,
                [&](uint32_t a, uint32_t b, uint32_t cc) { return Wr[a] * (X1r[b] * Gr[cc]); },
                [&](int k2, float acc) {
                    if constexpr (SHARED) {
                        const float s = bw_wave_sum(acc);
                        if (lane == 0) ws_x2[(tile * N + n) * nc2 + k2] = s;
                    } else {
                        GX2r[k2] = acc;
                    }
                });
        __syncthreads();  // the x1 rows have been read by every wave
        // gx1 into the x1 rows
        bw_pass(seg1, list1, k1b, k1e, lane,
                [&](uint32_t a, uint32_t b, uint32_t cc) { return X2r[b] * (Wr[a] * Gr[cc]); },
                [&](int k, float acc) { X1r[k] = acc; });
        __syncthreads();
        TIO* dst = gx1 + row0 * nc1;
        for (int e = tid; e < nch * nc1; e += kBw1wThreads) {
            const int r = e / nc1;
            const float v = X1[r * st1 + (e - r * nc1)];
            bw_store(dst + e, acc_gx1 ? bw_load(dst + e) + v : v);
        }
        if constexpr (!SHARED) {
            TIO* dst2 = gx2 + row0 * nc2;
            for (int e = tid; e < nch * nc2; e += kBw1wThreads) {
                const int r = e / nc2;
                bw_store(dst2 + e, GX2[r * st2 + (e - r * nc2)]);
            }
        }
    }
    __syncthreads();
    // the range's gW sums: 64 consecutive channels of a path per wave store
    if (n_end > n_begin)
        for (int i = tid; i < np * kBw1wLanes; i += kBw1wThreads) {
            const int p = i >> 6, r = i & 63;
            if (r < nch) ws_w[(group * np + p) * C + c0 + r] = GW[r * stw + p];
        }
}

// Forward: out[n,c,k3] = sum over the entries of k3 of W[c,p] T x1[n,c,k1] x2[.,k2]
// (the k3-ordered list), x2 per unit or (SHARED) one row per edge.  Same tiling as
// the gradients: a 64-channel tile and a range of edges per workgroup, the weight
// rows in LDS for the range, the four waves splitting the output slots.
// NV > 1 (SHARED only; the depthwise mode): NV second-input channels v of the edge
// at once, out[n,c,k3] = sum_v sum over the entries of W_v[c,p] T x1[n,c,k1] x2_v[n,k2]
// with the rows x2_v at x2 + n x2s + v x2v and the weight slices at wts + v wslice:
// each entry takes x1[k1] * sum_v W_v[p] x2_v[k2], so x1 and the list are read once
// for the NV channels and the output rows are stored once.
template <typename TIO, bool SHARED, int NV>
__global__ __launch_bounds__(kBw1wThreads) void spingtp_fwd_cw_kernel(
    const TIO* __restrict__ x1, const TIO* __restrict__ x2, const float* __restrict__ wts, TIO* __restrict__ out,
    int64_t N, int64_t C, int64_t epg, const uint32_t* __restrict__ tab, int64_t x2s, bool acc_out, int64_t x2v,
    int64_t wslice) {
    static_assert(NV >= 1 && (SHARED || NV == 1), "several second-input channels need the shared x2 form");
    extern __shared__ float lds[];
    const int nc1 = static_cast<int>(tab[0]), nc2 = static_cast<int>(tab[1]), nco = static_cast<int>(tab[2]);
    const int np = static_cast<int>(tab[3]);
    const uint32_t* __restrict__ seg3 = tab + tab[11];
    const uint32_t* __restrict__ list3 = tab + tab[12];
    const int stw = bw_stride(np), st1 = bw_stride(nc1), sto = bw_stride(nco), st2 = bw_stride(nc2);
    float* Wt = lds;                          // [NV][64][stw] weights of the tile's channels
    float* X1 = Wt + NV * kBw1wLanes * stw;   // [64][st1] x1 rows
    float* O = X1 + kBw1wLanes * st1;         // [64][sto] output rows
    float* X2 = O + kBw1wLanes * sto;         // [64][st2] x2 rows, or (SHARED) [NV][st2] the edge's x2 rows

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t group = blockIdx.x, tile = blockIdx.y;
    const int64_t c0 = tile * kBw1wLanes;
    const int nch = static_cast<int>(C - c0 < kBw1wLanes ? C - c0 : kBw1wLanes);
    const int64_t n_begin = group * epg;
    const int64_t n_end = n_begin + epg < N ? n_begin + epg : N;
    const uint32_t* __restrict__ kr = tab + 31;
    const int kb = static_cast<int>(kr[wave]), ke = static_cast<int>(kr[wave + 1]);

    const int total = kBw1wLanes * (NV * stw + st1 + sto) + (SHARED ? NV * st2 : kBw1wLanes * st2);
    for (int i = tid; i < total; i += kBw1wThreads) lds[i] = 0.f;
    __syncthreads();
#pragma unroll
    for (int v = 0; v < NV; ++v)
        for (int e = tid; e < nch * np; e += kBw1wThreads) {
            const int r = e / np;
            Wt[(v * kBw1wLanes + r) * stw + (e - r * np)] = wts[v * wslice + c0 * np + e];
        }
    const float* Wr = Wt + lane * stw;
    const float* X1r = X1 + lane * st1;
    const float* X2r = SHARED ? X2 : X2 + lane * st2;
    float* Or = O + lane * sto;

    for (int64_t n = n_begin; n < n_end; ++n) {
        __syncthreads();  // the previous edge's output rows have left
        const int64_t row0 = n * C + c0;
        bw_load_rows(x1 + row0 * nc1, nch, nc1, st1, X1, tid);
        if constexpr (SHARED) {
#pragma unroll
            for (int v = 0; v < NV; ++v)
                for (int k = tid; k < nc2; k += kBw1wThreads) X2[v * st2 + k] = bw_load(x2 + n * x2s + v * x2v + k);
        } else {
            bw_load_rows(x2 + row0 * nc2, nch, nc2, st2, X2, tid);
        }
        __syncthreads();
        bw_pass(
            seg3, list3, kb, ke, lane,
            [&](uint32_t a, uint32_t b, uint32_t cc) {
                if constexpr (NV == 1) {
                    return Wr[a] * (X1r[b] * X2r[cc]);
                } else {
                    float w2 = Wr[a] * X2r[cc];
#pragma unroll
                    for (int v = 1; v < NV; ++v) w2 = fmaf(Wr[v * kBw1wLanes * stw + a], X2r[v * st2 + cc], w2);
                    return X1r[b] * w2;
                }
            },
            [&](int k3, float acc) { Or[k3] = acc; });
        __syncthreads();
        TIO* dst = out + row0 * nco;
        for (int e = tid; e < nch * nco; e += kBw1wThreads) {
            const int r = e / nco;
            const float v = O[r * sto + (e - r * nco)];
            bw_store(dst + e, acc_out ? bw_load(dst + e) + v : v);
        }
    }
}

// gx2[n,k2] = sum over the channel tiles (fixed order)
template <typename TIO>
__global__ __launch_bounds__(256) void spingtp_bwd_v1w_reduce_x2_kernel(const float* __restrict__ ws_x2,
                                                                        TIO* __restrict__ gx2, int64_t nx2,
                                                                        int64_t tiles, int nc2, int64_t gx2s) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= nx2) return;
    float s = 0.f;
    for (int64_t t = 0; t < tiles; ++t) s += ws_x2[t * nx2 + i];
    const int64_t n = i / nc2;
    bw_store(gx2 + n * gx2s + (i - n * nc2), s);  // rows gx2s elements apart
}

// gW[c,p] = sum over the edge ranges: one workgroup per (path, 64 channels); wave w
// adds the ranges r = w, w + 16, ... (64 consecutive channels per load), and the 16
// wave sums are added in wave order.
constexpr int kBw1wReduceWaves = 16;

__global__ __launch_bounds__(64 * kBw1wReduceWaves) void spingtp_bwd_v1w_reduce_w_kernel(
    const float* __restrict__ ws_w, float* __restrict__ gw, int64_t C, int np, int64_t groups) {
    __shared__ float part[kBw1wReduceWaves][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t p = blockIdx.x, c = static_cast<int64_t>(blockIdx.y) * 64 + lane;
    float s = 0.f;
    if (c < C)
        for (int64_t r = wave; r < groups; r += kBw1wReduceWaves) s += ws_w[(r * np + p) * C + c];
    part[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && c < C) {
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < kBw1wReduceWaves; ++w) t += part[w][lane];
        gw[c * np + p] = t;
    }
}

// raise a kernel's dynamic LDS limit once per device (to the family's maximum); one
// flag set per (TIO, TAG), i.e. per kernel
template <typename TIO, int TAG>
hipError_t raise_lds_limit(const void* kernel) {
    constexpr int kMaxDevices = 64;
    static std::atomic<bool> raised[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    if (!raised[dev].load(std::memory_order_acquire)) {
        const hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 static_cast<int>(kBw1wMaxLdsFloats * sizeof(float)));
        if (e != hipSuccess) return e;
        raised[dev].store(true, std::memory_order_release);
    }
    return hipSuccess;
}

template <typename TIO, bool SHARED>
hipError_t launch_typed(const void* x1, const void* x2, const float* w, const void* g, void* gx1, void* gx2,
                        float* gw, float* ws, int64_t N, int64_t C, const Bw1wShape& s, const uint32_t* tab,
                        hipStream_t stream, int64_t x2s, bool acc_gx1) {
    const int64_t tiles = (C + kBw1wLanes - 1) / kBw1wLanes;
    int64_t groups = 0, epg = 0;
    bw1w_groups(N, C, &groups, &epg, bw_target_groups(SHARED ? s.lds_floats : s.lds_unit_bwd));
    float* ws_x2 = ws;
    float* ws_w = SHARED ? ws + tiles * N * s.nc2 : ws;
    if (groups > 0 && tiles > 0) {
        if (groups > 0x7fffffff || tiles > 0xffff) return hipErrorInvalidValue;
        const int lds_floats = SHARED ? s.lds_floats : s.lds_unit_bwd;
        const size_t bytes = static_cast<size_t>(lds_floats) * sizeof(float);
        if (bytes > 65536) {
            const hipError_t e = raise_lds_limit<TIO, SHARED ? 1 : 2>(
                reinterpret_cast<const void*>(&spingtp_bwd_v1w_kernel<TIO, SHARED>));
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL((spingtp_bwd_v1w_kernel<TIO, SHARED>),
                           dim3(static_cast<unsigned>(groups), static_cast<unsigned>(tiles)), dim3(kBw1wThreads), bytes,
                           stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2), w,
                           static_cast<const TIO*>(g), static_cast<TIO*>(gx1), static_cast<TIO*>(gx2), ws_x2, ws_w, N,
                           C, epg, tab, x2s, acc_gx1);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t nx2 = SHARED ? N * s.nc2 : 0;  // per-unit gx2 is written by the kernel
    if (nx2 > 0) {
        const int64_t blocks = (nx2 + 255) / 256;
        if (blocks > 0x7fffffff) return hipErrorInvalidValue;
        hipLaunchKernelGGL(spingtp_bwd_v1w_reduce_x2_kernel<TIO>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                           stream, ws_x2, static_cast<TIO*>(gx2), nx2, groups > 0 ? tiles : 0, s.nc2, x2s);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (C > 0 && s.np > 0) {  // zeros when there are no edges
        if (tiles > 0xffff) return hipErrorInvalidValue;
        hipLaunchKernelGGL(spingtp_bwd_v1w_reduce_w_kernel, dim3(static_cast<unsigned>(s.np), static_cast<unsigned>(tiles)),
                           dim3(64 * kBw1wReduceWaves), 0, stream, ws_w, gw, C, s.np, groups);
        return hipGetLastError();
    }
    return hipSuccess;
}

}  // namespace

void bw1w_groups(int64_t N, int64_t C, int64_t* groups, int64_t* epg, int target) {
    // about `target` workgroups over the channel tiles and edge ranges
    const int64_t tiles = (C + kBw1wLanes - 1) / kBw1wLanes;
    if (N <= 0 || tiles <= 0) {
        *groups = 0;
        *epg = 0;
        return;
    }
    int64_t want = target / tiles;
    if (want < 1) want = 1;
    if (want > N) want = N;
    *epg = (N + want - 1) / want;
    *groups = (N + *epg - 1) / *epg;
}

size_t bw1w_workspace_floats(int64_t N, int64_t C, const Bw1wShape& s) {
    int64_t groups = 0, epg = 0;
    bw1w_groups(N, C, &groups, &epg, bw_target_groups(s.lds_floats));  // as the launch splits them
    const int64_t tiles = (C + kBw1wLanes - 1) / kBw1wLanes;
    return static_cast<size_t>(tiles * N * s.nc2 + groups * s.np * C);
}

size_t bwcw_workspace_floats(int64_t N, int64_t C, const Bw1wShape& s) {
    int64_t groups = 0, epg = 0;
    bw1w_groups(N, C, &groups, &epg, bw_target_groups(s.lds_unit_bwd));  // as the launch splits them
    return static_cast<size_t>(groups * s.np * C);
}

hipError_t launch_bwd_v1w(int dtype, bool shared_x2, const void* x1, const void* x2, const float* w, const void* g,
                          void* gx1, void* gx2, float* gw, float* ws, int64_t N, int64_t C, const Bw1wShape& s,
                          const uint32_t* tab, hipStream_t stream, int64_t x2_stride, bool accumulate_gx1) {
    const int64_t x2s = x2_stride > 0 ? x2_stride : s.nc2;
    // the kernel carves its LDS from the table's sizes
    const int base = kBw1wLanes * (2 * bw_stride(s.np) + bw_stride(s.nc1) + bw_stride(s.nco));
    if (shared_x2) {
        if (s.lds_floats <= 0 || s.lds_floats > kBw1wMaxLdsFloats || s.lds_floats != base + bw_stride(s.nc2))
            return hipErrorInvalidValue;
        return dtype == 0
                   ? launch_typed<float, true>(x1, x2, w, g, gx1, gx2, gw, ws, N, C, s, tab, stream, x2s, accumulate_gx1)
                   : launch_typed<uint16_t, true>(x1, x2, w, g, gx1, gx2, gw, ws, N, C, s, tab, stream, x2s,
                                                  accumulate_gx1);
    }
    if (s.lds_unit_bwd <= 0 || s.lds_unit_bwd > kBw1wMaxLdsFloats ||
        s.lds_unit_bwd != base + 2 * kBw1wLanes * bw_stride(s.nc2))
        return hipErrorInvalidValue;
    return dtype == 0
               ? launch_typed<float, false>(x1, x2, w, g, gx1, gx2, gw, ws, N, C, s, tab, stream, x2s, accumulate_gx1)
               : launch_typed<uint16_t, false>(x1, x2, w, g, gx1, gx2, gw, ws, N, C, s, tab, stream, x2s,
                                               accumulate_gx1);
}

template <typename TIO, bool SHARED, int NV>
static hipError_t launch_fwd_typed(const void* x1, const void* x2, const float* w, void* out, int64_t N, int64_t C,
                                   int lds_floats, const uint32_t* tab, hipStream_t stream, int64_t x2s,
                                   bool acc_out, int64_t x2v, int64_t wslice) {
    const int64_t tiles = (C + kBw1wLanes - 1) / kBw1wLanes;
    int64_t groups = 0, epg = 0;
    bw1w_groups(N, C, &groups, &epg, bw_target_groups(lds_floats));
    if (groups == 0 || tiles == 0) return hipSuccess;
    if (groups > 0x7fffffff || tiles > 0xffff) return hipErrorInvalidValue;
    const size_t bytes = static_cast<size_t>(lds_floats) * sizeof(float);
    if (bytes > 65536) {
        const hipError_t e = raise_lds_limit<TIO, SHARED ? 3 + 2 * (NV - 1) : 4>(
            reinterpret_cast<const void*>(&spingtp_fwd_cw_kernel<TIO, SHARED, NV>));
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((spingtp_fwd_cw_kernel<TIO, SHARED, NV>),
                       dim3(static_cast<unsigned>(groups), static_cast<unsigned>(tiles)), dim3(kBw1wThreads), bytes,
                       stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2), w, static_cast<TIO*>(out), N,
                       C, epg, tab, x2s, acc_out, x2v, wslice);
    return hipGetLastError();
}

template <typename TIO>
static hipError_t launch_fwd_shared_nv(int nv, const void* x1, const void* x2, const float* w, void* out, int64_t N,
                                       int64_t C, int lds, const uint32_t* tab, hipStream_t stream, int64_t x2s,
                                       bool acc, int64_t x2v, int64_t wslice) {
    switch (nv) {
        case 1: return launch_fwd_typed<TIO, true, 1>(x1, x2, w, out, N, C, lds, tab, stream, x2s, acc, x2v, wslice);
        case 2: return launch_fwd_typed<TIO, true, 2>(x1, x2, w, out, N, C, lds, tab, stream, x2s, acc, x2v, wslice);
        case 3: return launch_fwd_typed<TIO, true, 3>(x1, x2, w, out, N, C, lds, tab, stream, x2s, acc, x2v, wslice);
        case 4: return launch_fwd_typed<TIO, true, 4>(x1, x2, w, out, N, C, lds, tab, stream, x2s, acc, x2v, wslice);
        default: return hipErrorInvalidValue;
    }
}

int fwd_cw_lds_floats(const Bw1wShape& s, int nv) {
    return s.lds_shared_fwd + (nv - 1) * (kBw1wLanes * bw_stride(s.np) + bw_stride(s.nc2));
}

hipError_t launch_fwd_cw(int dtype, bool shared_x2, const void* x1, const void* x2, const float* w, void* out,
                         int64_t N, int64_t C, const Bw1wShape& s, const uint32_t* tab, hipStream_t stream,
                         int64_t x2_stride, bool accumulate, int nv, int64_t x2v, int64_t wslice) {
    const int64_t x2s = x2_stride > 0 ? x2_stride : s.nc2;
    // the kernel carves its LDS from the table's sizes
    const int base = kBw1wLanes * (bw_stride(s.np) + bw_stride(s.nc1) + bw_stride(s.nco));
    const int lds1 = shared_x2 ? s.lds_shared_fwd : s.lds_unit_fwd;
    if (lds1 <= 0 || lds1 > kBw1wMaxLdsFloats ||
        lds1 != base + (shared_x2 ? bw_stride(s.nc2) : kBw1wLanes * bw_stride(s.nc2)))
        return hipErrorInvalidValue;
    if (nv < 1 || nv > kFwdCwMaxNv || (nv > 1 && !shared_x2)) return hipErrorInvalidValue;
    if (shared_x2) {
        const int lds = fwd_cw_lds_floats(s, nv);
        if (lds > kBw1wMaxLdsFloats) return hipErrorInvalidValue;
        return dtype == 0
                   ? launch_fwd_shared_nv<float>(nv, x1, x2, w, out, N, C, lds, tab, stream, x2s, accumulate, x2v, wslice)
                   : launch_fwd_shared_nv<uint16_t>(nv, x1, x2, w, out, N, C, lds, tab, stream, x2s, accumulate, x2v,
                                                    wslice);
    }
    return dtype == 0
               ? launch_fwd_typed<float, false, 1>(x1, x2, w, out, N, C, lds1, tab, stream, x2s, accumulate, 0, 0)
               : launch_fwd_typed<uint16_t, false, 1>(x1, x2, w, out, N, C, lds1, tab, stream, x2s, accumulate, 0, 0);
}

}  // namespace spingtp
