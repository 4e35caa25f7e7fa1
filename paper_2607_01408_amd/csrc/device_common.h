// Device helpers shared by the forward kernels: bf16 conversion, coalesced
// tile staging between HBM and LDS, and step (A) (coefficients -> theta-Fourier
// form of the three real polynomials of one input at one Gauss node).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "layout.h"

namespace spingtp {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);                                                     // nearest even
    return static_cast<uint16_t>(u >> 16);
}

template <int NC, int ST>
__device__ __forceinline__ void put(float* dst, int e, float v) {
    const int u = e / NC;
    dst[u * ST + (e - u * NC)] = v;
}

// Global tile (contiguous nvalid * NC elements, 256-byte aligned) -> LDS rows of stride ST.
template <int NC, int ST>
__device__ __forceinline__ void load_tile(const float* __restrict__ src, int nvalid, float* dst, int tid, int nthr) {
    const int n = nvalid * NC;
    const int n4 = n >> 2;
    const v4f* s4 = reinterpret_cast<const v4f*>(src);
    for (int i = tid; i < n4; i += nthr) {
        const v4f v = __builtin_nontemporal_load(s4 + i);
        const int e = 4 * i;
        put<NC, ST>(dst, e, v.x);
        put<NC, ST>(dst, e + 1, v.y);
        put<NC, ST>(dst, e + 2, v.z);
        put<NC, ST>(dst, e + 3, v.w);
    }
    for (int e = 4 * n4 + tid; e < n; e += nthr) put<NC, ST>(dst, e, src[e]);
}

template <int NC, int ST>
__device__ __forceinline__ void load_tile(const uint16_t* __restrict__ src, int nvalid, float* dst, int tid, int nthr) {
    const int n = nvalid * NC;
    const int n8 = n >> 3;
    const v4u* s8 = reinterpret_cast<const v4u*>(src);
    for (int i = tid; i < n8; i += nthr) {
        const v4u v = __builtin_nontemporal_load(s8 + i);
        const int e = 8 * i;
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            put<NC, ST>(dst, e + 2 * q, __uint_as_float(w[q] << 16));
            put<NC, ST>(dst, e + 2 * q + 1, __uint_as_float(w[q] & 0xffff0000u));
        }
    }
    for (int e = 8 * n8 + tid; e < n; e += nthr) put<NC, ST>(dst, e, bf16_to_f32(src[e]));
}

// Two full tiles (UNITS rows each): every 16-byte load of the thread is issued
// before the first LDS write, so the HBM latency is paid once, not per chunk.
template <int NC, int ST, int UNITS, int NTHR>
__device__ __forceinline__ void load_two_full_tiles(const float* __restrict__ a, const float* __restrict__ b,
                                                    float* da, float* db, int tid) {
    static_assert((UNITS * NC) % 4 == 0, "whole 16-byte chunks");
    constexpr int N4 = UNITS * NC / 4;
    constexpr int IT = (N4 + NTHR - 1) / NTHR;
    const v4f* a4 = reinterpret_cast<const v4f*>(a);
    const v4f* b4 = reinterpret_cast<const v4f*>(b);
    v4f ra[IT], rb[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N4) {
            ra[it] = __builtin_nontemporal_load(a4 + i);
            rb[it] = __builtin_nontemporal_load(b4 + i);
        }
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N4) {
            const int e = 4 * i;
            put<NC, ST>(da, e, ra[it].x);
            put<NC, ST>(da, e + 1, ra[it].y);
            put<NC, ST>(da, e + 2, ra[it].z);
            put<NC, ST>(da, e + 3, ra[it].w);
            put<NC, ST>(db, e, rb[it].x);
            put<NC, ST>(db, e + 1, rb[it].y);
            put<NC, ST>(db, e + 2, rb[it].z);
            put<NC, ST>(db, e + 3, rb[it].w);
        }
    }
}

template <int NC, int ST, int UNITS, int NTHR>
__device__ __forceinline__ void load_two_full_tiles(const uint16_t* __restrict__ a, const uint16_t* __restrict__ b,
                                                    float* da, float* db, int tid) {
    static_assert((UNITS * NC) % 8 == 0, "whole 16-byte chunks");
    constexpr int N8 = UNITS * NC / 8;
    constexpr int IT = (N8 + NTHR - 1) / NTHR;
    const v4u* a8 = reinterpret_cast<const v4u*>(a);
    const v4u* b8 = reinterpret_cast<const v4u*>(b);
    v4u ra[IT], rb[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N8) {
            ra[it] = __builtin_nontemporal_load(a8 + i);
            rb[it] = __builtin_nontemporal_load(b8 + i);
        }
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N8) {
            const int e = 8 * i;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                put<NC, ST>(da, e + 2 * q, __uint_as_float(ra[it][q] << 16));
                put<NC, ST>(da, e + 2 * q + 1, __uint_as_float(ra[it][q] & 0xffff0000u));
                put<NC, ST>(db, e + 2 * q, __uint_as_float(rb[it][q] << 16));
                put<NC, ST>(db, e + 2 * q + 1, __uint_as_float(rb[it][q] & 0xffff0000u));
            }
        }
    }
}

// One full tile (UNITS rows), every 16-byte load of the thread issued before the first
// LDS write (load_two_full_tiles for a single input).
template <int NC, int ST, int UNITS, int NTHR>
__device__ __forceinline__ void load_full_tile(const float* __restrict__ a, float* da, int tid) {
    static_assert((UNITS * NC) % 4 == 0, "whole 16-byte chunks");
    constexpr int N4 = UNITS * NC / 4;
    constexpr int IT = (N4 + NTHR - 1) / NTHR;
    const v4f* a4 = reinterpret_cast<const v4f*>(a);
    v4f ra[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N4) ra[it] = __builtin_nontemporal_load(a4 + i);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N4) {
            const int e = 4 * i;
            put<NC, ST>(da, e, ra[it].x);
            put<NC, ST>(da, e + 1, ra[it].y);
            put<NC, ST>(da, e + 2, ra[it].z);
            put<NC, ST>(da, e + 3, ra[it].w);
        }
    }
}

template <int NC, int ST, int UNITS, int NTHR>
__device__ __forceinline__ void load_full_tile(const uint16_t* __restrict__ a, float* da, int tid) {
    static_assert((UNITS * NC) % 8 == 0, "whole 16-byte chunks");
    constexpr int N8 = UNITS * NC / 8;
    constexpr int IT = (N8 + NTHR - 1) / NTHR;
    const v4u* a8 = reinterpret_cast<const v4u*>(a);
    v4u ra[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N8) ra[it] = __builtin_nontemporal_load(a8 + i);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int i = tid + it * NTHR;
        if (it < IT - 1 || i < N8) {
            const int e = 8 * i;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                put<NC, ST>(da, e + 2 * q, __uint_as_float(ra[it][q] << 16));
                put<NC, ST>(da, e + 2 * q + 1, __uint_as_float(ra[it][q] & 0xffff0000u));
            }
        }
    }
}

// Tile of an input shared by groups of cpx consecutive units (edge multiplicity
// one: unit u reads row u / cpx of src).  One wave per row, coalesced along the row;
// a wave issues the loads of four rows before their LDS writes (rows past nvalid
// repeat the last valid one and are not written), and the tile's first edge comes
// from one division.
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }

template <int NC, int ST, typename TIO>
__device__ __forceinline__ void load_tile_shared(const TIO* __restrict__ src, int64_t u0, int nvalid, int64_t cpx,
                                                 float* dst, int tid, int nthr) {
    constexpr int CI = (NC + 63) / 64;  // loads per row and lane
    constexpr int RB = 4;               // rows in flight per wave
    const int64_t n0 = u0 / cpx, r0 = u0 - n0 * cpx;  // the tile's first edge, its first channel
    const int waves = nthr >> 6, lane = tid & 63;
    for (int rb = tid >> 6; rb < nvalid; rb += RB * waves) {
        float v[RB][CI];
#pragma unroll
        for (int i = 0; i < RB; ++i) {
            const int r = rb + i * waves < nvalid ? rb + i * waves : nvalid - 1;
            const TIO* __restrict__ s = src + (n0 + (r0 + r) / cpx) * NC;
#pragma unroll
            for (int j = 0; j < CI; ++j) {
                const int c = lane + 64 * j;
                v[i][j] = c < NC ? to_f32(s[c]) : 0.f;
            }
        }
#pragma unroll
        for (int i = 0; i < RB; ++i) {
            const int r = rb + i * waves;
            if (r < nvalid) {
#pragma unroll
                for (int j = 0; j < CI; ++j) {
                    const int c = lane + 64 * j;
                    if (c < NC) dst[r * ST + c] = v[i][j];
                }
            }
        }
    }
}

// Both input tiles of a workgroup: the batched path for full tiles, the
// element-exact loop for the ragged last tile.
template <int NC, int ST, int UNITS, int NTHR, typename TIO>
__device__ __forceinline__ void load_two_tiles(const TIO* __restrict__ a, const TIO* __restrict__ b, int nvalid,
                                               float* da, float* db, int tid) {
    if (nvalid == UNITS) {
        load_two_full_tiles<NC, ST, UNITS, NTHR>(a, b, da, db, tid);
    } else {
        load_tile<NC, ST>(a, nvalid, da, tid, NTHR);
        load_tile<NC, ST>(b, nvalid, db, tid, NTHR);
    }
}

template <int NC, int ST>
__device__ __forceinline__ float get(const float* src, int e) {
    const int u = e / NC;
    return src[u * ST + (e - u * NC)];
}

template <int NC, int ST>
__device__ __forceinline__ void store_tile(float* __restrict__ dst, int nvalid, const float* src, int tid, int nthr) {
    const int n = nvalid * NC;
    const int n4 = n >> 2;
    v4f* d4 = reinterpret_cast<v4f*>(dst);
    for (int i = tid; i < n4; i += nthr) {
        const int e = 4 * i;
        v4f v;
        v.x = get<NC, ST>(src, e);
        v.y = get<NC, ST>(src, e + 1);
        v.z = get<NC, ST>(src, e + 2);
        v.w = get<NC, ST>(src, e + 3);
        __builtin_nontemporal_store(v, d4 + i);
    }
    for (int e = 4 * n4 + tid; e < n; e += nthr) dst[e] = get<NC, ST>(src, e);
}

template <int NC, int ST>
__device__ __forceinline__ void store_tile(uint16_t* __restrict__ dst, int nvalid, const float* src, int tid, int nthr) {
    const int n = nvalid * NC;
    const int n8 = n >> 3;
    v4u* d8 = reinterpret_cast<v4u*>(dst);
    for (int i = tid; i < n8; i += nthr) {
        const int e = 8 * i;
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            w[q] = static_cast<uint32_t>(f32_to_bf16(get<NC, ST>(src, e + 2 * q))) |
                   (static_cast<uint32_t>(f32_to_bf16(get<NC, ST>(src, e + 2 * q + 1))) << 16);
        const v4u v = {w[0], w[1], w[2], w[3]};
        __builtin_nontemporal_store(v, d8 + i);
    }
    for (int e = 8 * n8 + tid; e < n; e += nthr) dst[e] = f32_to_bf16(get<NC, ST>(src, e));
}

// Parity-labelled basis (paper Sec. 3.4 eq. parity_basis): in a tile of rows
// [spin -1 | 0 | +1][(L+1)^2] at stride st, map parity-basis coefficients to the
// real basis the kernels compute in (x = P x_p; inverse = false) or real-basis
// outputs back to the parity basis (y_p = P^T y; inverse = true).  Per slot of
// degree l >= 1 of the -1 and +1 blocks (c_+ stored in the -1 block, c_- in +1):
// x[-1] = (c_+ + c_-)/sqrt2, x[+1] = (-1)^l (c_+ - c_-)/sqrt2.
template <int L>
__device__ void parity_mix_rows(float* tile, int st, int rows, bool inverse, int tid, int nthr) {
    constexpr int B = (L + 1) * (L + 1);
    constexpr int NQ = B - 1;  // slots with l >= 1 in one spin block
    const float h = 0.70710678118654752440f;
    for (int i = tid; i < rows * NQ; i += nthr) {
        const int r = i / NQ, q = i - r * NQ + 1;
        int l = 0;  // degree of slot q: the number of k >= 1 with k^2 <= q
#pragma unroll
        for (int k = 1; k <= L; ++k) l += q >= k * k ? 1 : 0;
        const float t = (l & 1) ? -1.f : 1.f;
        float* row = tile + static_cast<int64_t>(r) * st;
        const float a = row[q], b = row[2 * B + q];
        if (!inverse) {
            row[q] = (a + b) * h;
            row[2 * B + q] = t * (a - b) * h;
        } else {
            row[q] = fmaf(t, b, a) * h;
            row[2 * B + q] = fmaf(-t, b, a) * h;
        }
    }
}

// Step (A) for one input of degree L at one theta node.
//   xr  : this lane's LDS row ([n_spins][(L+1)^2], spin order -1, 0, +1)
//   tb  : the node's table block; n0: the global N0 mixing of input 1, followed by
//         that of input 2 (equal except in the tables of spingtp_backward);
//   second: this lane transforms input 2.
//   PAR : the row holds parity-basis coefficients; the |s| = 1 blocks are mixed by
//         P as they are read (the kernels that stage tiles in LDS mix them there
//         instead and pass false).
//   FENCE: a scheduling barrier after each order t of the |s| = 1 sums and after
//         the s = 0 sums, so that the compiler keeps only one order's row values
//         in flight (for callers that hold other live state across this step).
template <int L, int LA, bool SPIN, bool PAR = false, bool FENCE = false>
__device__ __forceinline__ void coef_to_theta_fourier(const float* xr, const float* __restrict__ tb,
                                                      const float* __restrict__ n0, bool second, float (&Ac)[L + 1],
                                                      float (&As)[L + 1], float (&Bc)[L + 1], float (&Bs)[L + 1],
                                                      float (&Cc)[L + 1], float (&Cs)[L + 1], float& dl, float& ep) {
    constexpr Layout Y = make_layout(LA, 0, 0);  // only the per-node A offsets are used
    constexpr int B = (L + 1) * (L + 1);
    const float* x0 = xr + (SPIN ? B : 0);
#pragma unroll
    for (int t = 0; t <= L; ++t) {
        float sc = 0.f, ss = 0.f;
#pragma unroll
        for (int l = t; l <= L; ++l) {
            sc = fmaf(x0[l * l + l + t], tb[Y.a0c + tri(LA, t, l)], sc);
            if (t > 0) ss = fmaf(x0[l * l + l - t], tb[Y.a0s + tri(LA, t, l)], ss);
        }
        Ac[t] = sc;
        As[t] = ss;
    }
    if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);
    if constexpr (SPIN) {
        const float* xm = xr;
        const float* xp = xr + 2 * B;
        // paper-basis -1 and +1 values of slot q (degree l), up to the factor hs: with
        // c_+ stored in the -1 block and c_- in the +1 block, x[-1] = (c_+ + c_-)/sqrt2
        // and x[+1] = (-1)^l (c_+ - c_-)/sqrt2
        auto vm_of = [&](int q) { return PAR ? xm[q] + xp[q] : xm[q]; };
        auto vp_of = [&](int q, int l) { return PAR ? ((l & 1) ? xp[q] - xm[q] : xm[q] - xp[q]) : xp[q]; };
        const float hs = PAR ? 0.70710678118654752440f : 1.f;
#pragma unroll
        for (int t = 1; t <= L; ++t) {
            float up = 0.f, vp = 0.f, um = 0.f, vm = 0.f;
#pragma unroll
            for (int l = t; l <= L; ++l) {
                const float wp = tb[Y.aup + tri(LA, t, l)];
                const float wm = tb[Y.aum + tri(LA, t, l)];
                up = fmaf(vp_of(l * l + l + t, l), wp, up);
                vp = fmaf(vp_of(l * l + l - t, l), wp, vp);
                um = fmaf(vm_of(l * l + l + t), wm, um);
                vm = fmaf(vm_of(l * l + l - t), wm, vm);
            }
            if constexpr (PAR) up *= hs, vp *= hs, um *= hs, vm *= hs;
            Bc[t] = up + um;
            Bs[t] = -(vp + vm);
            Cc[t] = vp - vm;
            Cs[t] = up - um;
            if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);
        }
        float wpl = 0.f, wmi = 0.f;
#pragma unroll
        for (int l = 1; l <= L; ++l) {
            const float w = tb[Y.aw + l];
            wpl = fmaf(vp_of(l * l + l, l), w, wpl);
            wmi = fmaf(vm_of(l * l + l), w, wmi);
        }
        if constexpr (PAR) wpl *= hs, wmi *= hs;
        float c[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) c[i] = second ? n0[8 + i] : n0[i];
        Bc[0] = fmaf(c[0], wpl, c[1] * wmi);
        Cc[0] = fmaf(c[2], wpl, c[3] * wmi);
        dl = fmaf(c[4], wpl, c[5] * wmi);
        ep = fmaf(c[6], wpl, c[7] * wmi);
        Bs[0] = 0.f;
        Cs[0] = 0.f;
    } else {
        dl = ep = 0.f;
    }
}

}  // namespace
}  // namespace spingtp
