// Matrix-core SpinGTP forward kernel for L1 = L2 = Lout = L, spins {-1, 0, +1},
// on gfx950 (CDNA4).
//
// The five steps are those of the vector-ALU kernel (paper App. B, proof of the
// runtime proposition; Sec. 3.2 eq. generalized_gaunt): (A) theta-Fourier form
// of the six real trigonometric polynomials (three per input) at a Gauss node,
// (B) synthesis at the n_phi uniform points, (C) the three product combinations,
// (D) analysis onto cos/sin(t phi), (E) projection onto the output coefficients
// with the node's weight.  Steps (B) and (D) -- two thirds of the arithmetic --
// are contractions with tables shared by every unit, so they run as fp16
// matrix-core products with fp32 accumulation, the unit index being the N
// dimension of v_mfma_f32_32x32x16_f16:
//   (B)  field[point, unit] = TB[point, kappa] * F[kappa, unit]
//   (D)  spec[row, unit]    = TD[row, point]   * H[point, unit]
// kappa runs over the 16 coefficient slots of one polynomial (cos t = 0..L at
// 0..7, sin t at 8 + t); rows of (D) are cos/sin spectra t' = 0..L.
//
// Precision.  For fp32 I/O every operand is split into fp16 high and low parts
// and each product is hi*hi + hi*lo + lo*hi (each exact in the fp32 accumulator),
// which leaves a relative error near 2^-20 per term -- fp32-like.  bf16 I/O uses
// the high parts only (2^-11).  fp16 has a narrow exponent range, so each input
// row of every unit is first scaled by a power of two that puts its largest
// magnitude in [1/2, 1); by Cauchy-Schwarz every field is then bounded by
// sqrt(sum_lm |Y_lm|^2 * n_coef) < 64 and every product combination by < 2^14,
// well inside fp16, and the output is scaled back exactly.
//
// Work mapping.  A workgroup has four waves (one per SIMD, two workgroups per
// CU).  Up to L = 6 it owns 64 units: wave w takes units 32 (w & 1) .. +31 and the
// Gauss nodes j = (w >> 1) + 2k.  At L = 7, 8 two fp32 64-unit tiles would need
// more than half the LDS, so a workgroup owns 32 units and wave w takes the nodes
// j = w + 4k (NG = 4 node groups).  In a wave, lane u (< 32)
// works on input 1 and lane u + 32 on input 2 of unit u in step (A); a
// half-wave swap (v_permlane32_swap) then
// turns the two halves into the (B) operands, whose K layout puts kappa 0..7 in
// lanes 0..31 and 8..15 in lanes 32..63.  The (B) accumulator of lane u + 32h
// holds rows (points) 8i + 4h + r, so the products are lane-local, and the same
// registers, re-split, are the (D) operand.  The (D) tables put the cosine rows
// of R0 and P1 and the sine rows of P2 in the h = 0 accumulator positions and the
// other type in h = 1 (row t' = 0 is cos 0 in both), so every lane forms its
// output slots from its own registers: the h = 0 half accumulates the m3 >= 0
// outputs and the h = 1 half the m3 < 0 outputs (plus the m3 = 0, s3 = -1 ones),
// over its nodes, with table values that are the same for all 64 lanes (scalar
// loads).  The waves of a unit tile add their partial outputs in LDS at the end,
// in a fixed order (with four node groups, groups 2 and 3 write two tiles and
// groups 0 and 1 then add into them).
//
// L = 8 needs 17 coefficient slots per polynomial: sin 8 takes the slot sin 0
// leaves free and cos 8 goes into a second step-(B) K block, whose operand holds
// each lane's own cos 8 (input 1 at kappa 16, input 2 at kappa 24 -- no swap) and
// whose two tables each keep one of the two.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace spingtp {
namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

template <int L>
struct MShape {
    static constexpr Layout Y = make_layout(L, L, L);
    static constexpr int NT = Y.NT;
    static constexpr int NP = Y.NP;
    static constexpr int BLK = (L + 1) * (L + 1);
    static constexpr int NC = 3 * BLK;
    static constexpr int ST = NC | 1;           // odd row stride: conflict-free per-lane row reads
    // Two workgroups of four waves per CU (two waves per SIMD): 64-unit tiles (two
    // unit tiles of 32, two node groups) while two fp32 64-unit tiles fit half the
    // LDS, else (L >= 7) 32-unit tiles (one unit tile, four node groups).
    static constexpr bool WIDE = (2 * 64 * ST + 32 + 2 * 64) * 4 > 80 * 1024;
    static constexpr int UNITS = WIDE ? 32 : 64;
    static constexpr int UT = UNITS / 32;         // unit tiles of a workgroup
    static constexpr int X2 = UNITS * ST + 32;  // input-2 tile: lane u + 32 reads 32 banks away from lane u
    static constexpr int XF = X2 + UNITS * ST;
    static constexpr int YB = UNITS * ST;       // second partial-output tile (the first is at 0)
    static constexpr int REGION = XF > 2 * YB ? XF : 2 * YB;
    static constexpr int SCALE = REGION;        // 2 x UNITS power-of-two exponents
    static constexpr int LDS_FLOATS = REGION + 2 * UNITS;
    static constexpr int NB = (NP + 15) / 16;   // K blocks of step (D)
    static constexpr int KB = L >= 8 ? 2 : 1;   // K blocks of step (B): cos 8 in the second
    static constexpr int WAVES = 4;
    static constexpr int THREADS = 64 * WAVES;
    static constexpr int NG = WAVES / UT;         // node groups: wave w takes nodes w/UT, w/UT + NG, ...
    static constexpr int NPW = (NT + NG - 1) / NG;  // nodes per wave (at most)
    static constexpr int TB_WORDS = 64 * 8;     // one lane: 4 words hi, 4 words lo
    static_assert(L >= 1 && L <= 8, "cos 0..7 and sin 1..8 share the first K block; only cos 8 takes a second");
    static_assert(NP <= 32, "the phi points must fit the 32 rows of one step-(B) tile");
    static_assert(NT >= NG, "every wave takes at least one node");
    static_assert(LDS_FLOATS * 4 <= 80 * 1024, "two workgroups per CU");
    // step-(B) accumulator position v holds point 8 (v/4) + 4h + v%4; it carries a
    // point (for h = 0, hence possibly for h = 1) when that row is < n_phi
    __host__ __device__ static constexpr bool holds_point(int v) { return 8 * (v / 4) + (v % 4) < NP; }
};

__device__ __forceinline__ float swap_adjacent(float v) {
    // quad_perm [1,0,3,2]: value of the neighbouring lane (all lanes active)
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

// (a, b) split as fp16 hi + lo: hw = (fp16(a), fp16(b)) rounded toward zero,
// lw = (fp16(a - hi_a), fp16(b - hi_b)) rounded to nearest; each residual is exact
// in fp32 and below one fp16 unit of the value, so |x - hi - lo| <= 2^-21 |x| for
// normal x.
//
// Four instructions a pair, all the compiler's own (its hazard model sees every
// write; no inline asm, which its wait-state counting takes for one instruction
// whatever it holds).  The high word comes from the v_cvt_pkrtz intrinsic and the
// residuals from that word's own bits: a plain fp16 conversion would let the
// compiler fold the FMA that produced a value into the conversion (one rounding
// of the exact result) while forming the residual from the fp32-rounded value,
// and where those two roundings differ hi + lo misses the value by one fp16 unit.
// Each residual is fma(hi, m, a) with m = -1 passed in at run time: the compiler
// cannot fold the product away, so it reads the fp16 half straight from the packed
// word (v_fma_mix_f32, op_sel) instead of converting it first.  a - hi is exact in
// fp32, so the residual equals a - hi bit for bit.
__device__ __forceinline__ void split_pair(float a, float b, float m, uint32_t& hw, uint32_t& lw) {
    const h2 hq = __builtin_bit_cast(h2, __builtin_amdgcn_cvt_pkrtz(a, b));
    hw = __builtin_bit_cast(uint32_t, hq);
    const h2 lp = {static_cast<_Float16>(__builtin_fmaf(static_cast<float>(hq.x), m, a)),
                   static_cast<_Float16>(__builtin_fmaf(static_cast<float>(hq.y), m, b))};
    lw = __builtin_bit_cast(uint32_t, lp);
}

__device__ __forceinline__ uint32_t pack_hi(float a, float b) {
    const h2 hp = {static_cast<_Float16>(a), static_cast<_Float16>(b)};
    return __builtin_bit_cast(uint32_t, hp);
}

// Eight values (v[0..7]; zero where !live) -> hi and (SPLIT == 3) lo operands;
// m = -1 (see split_pair).
template <int SPLIT>
__device__ __forceinline__ void split8(const float (&v)[8], const bool (&live)[8], float m, v8h& hi, v8h& lo) {
    v4u h, l;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        if (!live[2 * w] && !live[2 * w + 1]) {
            h[w] = 0u;
            l[w] = 0u;
        } else if constexpr (SPLIT == 3) {
            uint32_t hw, lw;
            split_pair(v[2 * w], v[2 * w + 1], m, hw, lw);
            h[w] = hw;
            l[w] = lw;
        } else {
            h[w] = pack_hi(v[2 * w], v[2 * w + 1]);
            l[w] = 0u;
        }
    }
    hi = __builtin_bit_cast(v8h, h);
    lo = __builtin_bit_cast(v8h, l);
}

// v_permlane32_swap: exchanges the upper half-wave of a with the lower half-wave of b.
__device__ __forceinline__ void permlane32_swap(uint32_t a, uint32_t b, uint32_t& r0, uint32_t& r1) {
    const auto r = __builtin_amdgcn_permlane32_swap(a, b, false, false);
    r0 = r[0];
    r1 = r[1];
}

// (a, b) -> (a with its upper half-wave replaced by b's lower half,
//            b with its lower half-wave replaced by a's upper half)
__device__ __forceinline__ void swap_halves(const v8h& a, const v8h& b, v8h& r0, v8h& r1) {
    const v4u ua = __builtin_bit_cast(v4u, a), ub = __builtin_bit_cast(v4u, b);
    v4u o0, o1;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        uint32_t x, y;
        permlane32_swap(ua[w], ub[w], x, y);
        o0[w] = x;
        o1[w] = y;
    }
    r0 = __builtin_bit_cast(v8h, o0);
    r1 = __builtin_bit_cast(v8h, o1);
}

// Value of lanes 0..31 (lo) and of lanes 32..63 (hi) of x, in every lane.
__device__ __forceinline__ void bcast_halves(float x, float& lo, float& hi) {
    uint32_t a, b;
    permlane32_swap(__float_as_uint(x), __float_as_uint(x), a, b);
    lo = __uint_as_float(a);
    hi = __uint_as_float(b);
}

__device__ __forceinline__ v16f mfma(const v8h& a, const v8h& b, const v16f& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Output tile = partial tile A + partial tile B (row stride ST), coalesced
// 16-byte stores.  Full tiles: all LDS reads of a thread are issued before its
// first store, so the LDS latency is paid once.
template <int NC, int ST>
__device__ __forceinline__ int lds_off(int e) {
    if constexpr (ST == NC) {
        return e;
    } else {
        const int u = e / NC;
        return u * ST + (e - u * NC);
    }
}

template <int NC, int ST, int VEC>
__device__ __forceinline__ void gather_sum(const float* lds, int yb, int e, float (&v)[VEC]) {
#pragma unroll
    for (int q = 0; q < VEC; ++q) {
        const int o = lds_off<NC, ST>(e + q);
        v[q] = lds[o] + lds[yb + o];
    }
}

template <int NC, int ST, int UNITS, int NTHR>
__device__ __forceinline__ void store_out(float* __restrict__ dst, int nvalid, const float* lds, int yb, int tid) {
    v4f* d4 = reinterpret_cast<v4f*>(dst);
    if (nvalid == UNITS) {
        static_assert((UNITS * NC) % 4 == 0, "whole 16-byte chunks");
        constexpr int N4 = UNITS * NC / 4;
        constexpr int IT = (N4 + NTHR - 1) / NTHR;
        float v[IT][4];
#pragma unroll
        for (int it = 0; it < IT; ++it)
            if (it < IT - 1 || tid + it * NTHR < N4) gather_sum<NC, ST, 4>(lds, yb, 4 * (tid + it * NTHR), v[it]);
#pragma unroll
        for (int it = 0; it < IT; ++it)
            if (it < IT - 1 || tid + it * NTHR < N4) {
                const v4f w = {v[it][0], v[it][1], v[it][2], v[it][3]};
                __builtin_nontemporal_store(w, d4 + tid + it * NTHR);
            }
        return;
    }
    const int n = nvalid * NC;
    const int n4 = n >> 2;
    for (int i = tid; i < n4; i += NTHR) {
        float v[4];
        gather_sum<NC, ST, 4>(lds, yb, 4 * i, v);
        const v4f w = {v[0], v[1], v[2], v[3]};
        __builtin_nontemporal_store(w, d4 + i);
    }
    for (int e = 4 * n4 + tid; e < n; e += NTHR) {
        const int o = lds_off<NC, ST>(e);
        dst[e] = lds[o] + lds[yb + o];
    }
}

__device__ __forceinline__ uint32_t bf16x2(float a, float b) {
    return static_cast<uint32_t>(f32_to_bf16(a)) | (static_cast<uint32_t>(f32_to_bf16(b)) << 16);
}

template <int NC, int ST, int UNITS, int NTHR>
__device__ __forceinline__ void store_out(uint16_t* __restrict__ dst, int nvalid, const float* lds, int yb, int tid) {
    v4u* d8 = reinterpret_cast<v4u*>(dst);
    if (nvalid == UNITS) {
        static_assert((UNITS * NC) % 8 == 0, "whole 16-byte chunks");
        constexpr int N8 = UNITS * NC / 8;
        constexpr int IT = (N8 + NTHR - 1) / NTHR;
        float v[IT][8];
#pragma unroll
        for (int it = 0; it < IT; ++it)
            if (it < IT - 1 || tid + it * NTHR < N8) gather_sum<NC, ST, 8>(lds, yb, 8 * (tid + it * NTHR), v[it]);
#pragma unroll
        for (int it = 0; it < IT; ++it)
            if (it < IT - 1 || tid + it * NTHR < N8) {
                const v4u w = {bf16x2(v[it][0], v[it][1]), bf16x2(v[it][2], v[it][3]), bf16x2(v[it][4], v[it][5]),
                               bf16x2(v[it][6], v[it][7])};
                __builtin_nontemporal_store(w, d8 + tid + it * NTHR);
            }
        return;
    }
    const int n = nvalid * NC;
    const int n8 = n >> 3;
    for (int i = tid; i < n8; i += NTHR) {
        float v[8];
        gather_sum<NC, ST, 8>(lds, yb, 8 * i, v);
        const v4u w = {bf16x2(v[0], v[1]), bf16x2(v[2], v[3]), bf16x2(v[4], v[5]), bf16x2(v[6], v[7])};
        __builtin_nontemporal_store(w, d8 + i);
    }
    for (int e = 8 * n8 + tid; e < n; e += NTHR) {
        const int o = lds_off<NC, ST>(e);
        dst[e] = f32_to_bf16(lds[o] + lds[yb + o]);
    }
}

// SPLIT = 3: hi*hi + hi*lo + lo*hi (fp32 I/O); SPLIT = 1: hi*hi (bf16 I/O).
template <int L, typename TIO, int SPLIT, bool BWD>
__global__ __launch_bounds__(MShape<L>::THREADS, 2) void spingtp_fwd_mfma_kernel(const TIO* __restrict__ x1,
                                                                   const TIO* __restrict__ x2,
                                                                   TIO* __restrict__ out, int64_t units,
                                                                   int64_t cpx2, const float* __restrict__ tab,
                                                                   const uint32_t* __restrict__ aux,
                                                                   float neg_one) {
    using S = MShape<L>;
    constexpr Layout Y = S::Y;
    constexpr int NC = S::NC, ST = S::ST, BLK = S::BLK, NB = S::NB;
    __shared__ float lds[S::LDS_FLOATS];
    int* ex = reinterpret_cast<int*>(lds + S::SCALE);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t u0 = static_cast<int64_t>(blockIdx.x) * S::UNITS;
    const int nvalid = static_cast<int>(units - u0 < S::UNITS ? units - u0 : S::UNITS);

    // (1) input tiles -> LDS; rows past the end of the batch are zero
    if (cpx2 == 1) {
        load_two_tiles<NC, ST, S::UNITS, S::THREADS>(x1 + u0 * NC, x2 + u0 * NC, nvalid, lds, lds + S::X2, tid);
    } else {  // x2 shared by the cpx2 channels of an edge
        if (nvalid == S::UNITS) load_full_tile<NC, ST, S::UNITS, S::THREADS>(x1 + u0 * NC, lds, tid);
        else load_tile<NC, ST>(x1 + u0 * NC, nvalid, lds, tid, S::THREADS);
        load_tile_shared<NC, ST>(x2, u0, nvalid, cpx2, lds + S::X2, tid, S::THREADS);
    }
    for (int i = tid; i < (S::UNITS - nvalid) * ST; i += S::THREADS) {
        lds[nvalid * ST + i] = 0.f;
        lds[S::X2 + nvalid * ST + i] = 0.f;
    }
    __syncthreads();
    const bool parity = tab[Y.par] != 0.f;  // uniform

    // (2) per unit and input: scale the row by 2^-e so that its largest valid
    //     magnitude is in [1/2, 1).  Two threads per row (four with 32-unit tiles,
    //     outside the parity basis); the l = 0 slots of the |s| = 1 sectors are not
    //     data and are skipped.
    if (S::WIDE && !parity) {
        constexpr int Q = (NC + 3) / 4;
        const int row = tid >> 2;  // 0..2 UNITS - 1, the four threads of a row in one quad
        const int part = tid & 3;
        float* xr = lds + (row >= S::UNITS ? S::X2 : 0) + (row % S::UNITS) * ST + part * Q;
        float v[Q];
        float m = 0.f;
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            const int q = part * Q + i;
            v[i] = q < NC ? xr[i] : 0.f;
            m = fmaxf(m, (q == 0 || q == 2 * BLK) ? 0.f : fabsf(v[i]));
        }
        m = fmaxf(m, swap_adjacent(m));
        m = fmaxf(m, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(m), 0x4E, 0xF, 0xF, false)));
        int e = 0;
        if (m > 0.f && m <= 3.0e38f) (void)frexpf(m, &e);
        e = e < -100 ? -100 : (e > 100 ? 100 : e);
#pragma unroll
        for (int i = 0; i < Q; ++i)
            if (part * Q + i < NC) xr[i] = ldexpf(v[i], -e);
        if (part == 0) ex[row] = e;
    } else if (tid < 4 * S::UNITS) {  // two threads per row
        constexpr int HALF = (NC + 1) / 2;
        const int row = tid >> 1;  // 0..2 UNITS - 1: input row / UNITS, unit row % UNITS
        const bool odd = (tid & 1) != 0;
        float* xr = lds + (row >= S::UNITS ? S::X2 : 0) + (row % S::UNITS) * ST + (odd ? HALF : 0);
        float v[HALF];
        float m = 0.f;
#pragma unroll
        for (int i = 0; i < HALF; ++i) {
            const bool last = i + HALF >= NC;  // past the row end in the second half
            v[i] = (last && odd) ? 0.f : xr[i];
        }
        if (parity) {
            // parity-labelled basis: slot q of the s = -1 block (first half, v[q]) and
            // of the s = +1 block (second half, v[2 BLK + q - HALF]) become
            // ((a + b)/sqrt2, (-1)^l (a - b)/sqrt2), a = x[q], b = x[2 BLK + q]
#pragma unroll
            for (int l = 1; l <= L; ++l)
#pragma unroll
                for (int q = l * l; q < (l + 1) * (l + 1); ++q) {
                    const float mine = odd ? v[2 * BLK + q - HALF] : v[q];
                    const float other = swap_adjacent(mine);
                    const float a = odd ? other : mine, b = odd ? mine : other;
                    if (odd)
                        v[2 * BLK + q - HALF] = ((l & 1) ? (b - a) : (a - b)) * 0.70710678118654752440f;
                    else
                        v[q] = (a + b) * 0.70710678118654752440f;
                }
        }
#pragma unroll
        for (int i = 0; i < HALF; ++i) {
            bool skip = false;  // l = 0 slots of the s = -1 (index 0) and s = +1 (index 2 BLK) blocks
            if (i == 0) skip = !odd;
            if (i == 2 * BLK) skip = skip || !odd;
            if (i == 2 * BLK - HALF) skip = skip || odd;
            m = fmaxf(m, skip ? 0.f : fabsf(v[i]));
        }
        m = fmaxf(m, swap_adjacent(m));
        int e = 0;
        if (m > 0.f && m <= 3.0e38f) (void)frexpf(m, &e);
        e = e < -100 ? -100 : (e > 100 ? 100 : e);
#pragma unroll
        for (int i = 0; i < HALF; ++i) {
            const bool last = i + HALF >= NC;
            if (!(last && odd)) xr[i] = ldexpf(v[i], -e);
        }
        if (!odd) ex[row] = e;
    }
    __syncthreads();

    const int h = lane >> 5;  // (A): input h + 1; (D)-(E): accumulator type
    const int T = S::UT == 2 ? (wave & 1) : 0;       // unit tile of this wave
    // node group of this wave.  Where the nodes split evenly over the groups (L = 5, 6)
    // the assignment rotates from one workgroup to the next (by blockIdx / 256), which
    // measured 2-3 % faster (organic L = 6: fp32 8.41-8.53 against 8.68-8.78 ms, bf16
    // 6.45 against 6.59, alternated on one GPU); where they do not (L = 4, 7, 8) it
    // measured slower (catalyst +5 %, molecule +2 %) and is not applied.  Each group's
    // nodes and the fixed order in which the groups' partial outputs are summed do not
    // depend on the rotation, so the results are the same bit for bit.
    constexpr int ROT = S::NT % S::NG == 0 ? 1 : 0;
    const int ngrp = ((S::UT == 2 ? (wave >> 1) : wave) + ROT * static_cast<int>((blockIdx.x >> 8) % S::NG)) % S::NG;
    const float* xr = lds + (h ? S::X2 : 0) + (32 * T + (lane & 31)) * ST;
    const float sg = h ? -1.f : 1.f;
    const v4u* __restrict__ ops = reinterpret_cast<const v4u*>(aux);
    // The step-(B) operand tables of this lane: held in registers across the node loop,
    // except in the fp32 instantiations at L = 7, 8, whose registers run short: there
    // each node reads them again (L1-resident; offset by node x a zero the compiler
    // cannot see, so that the reads are not hoisted back out of the loop).  Measured on
    // 262,144 units: L = 8 0.565 -> 0.515 ms (63 -> 44 spilled VGPRs), L = 7 -2 %
    // (15 -> 0); at L = 6 fp32 and in bf16 the reads cost 1-2 %.
    constexpr bool RELOAD = SPLIT == 3 && L >= 7;
    constexpr int TB2 = 2 * 64 * (1 + 2 * NB);  // the second step-(B) blocks (L = 8), in v4u
    const int zero_i = static_cast<int>(neg_one + 1.0f);
    auto tables = [&](const v4u* __restrict__ o, v8h& h, v8h& l, v8h& ah, v8h& al, v8h& bh, v8h& bl) {
        h = __builtin_bit_cast(v8h, o[2 * lane]);
        l = __builtin_bit_cast(v8h, o[2 * lane + 1]);
        ah = S::KB == 2 ? __builtin_bit_cast(v8h, o[TB2 + 2 * lane]) : v8h{};
        al = S::KB == 2 ? __builtin_bit_cast(v8h, o[TB2 + 2 * lane + 1]) : v8h{};
        bh = S::KB == 2 ? __builtin_bit_cast(v8h, o[TB2 + 128 + 2 * lane]) : v8h{};
        bl = S::KB == 2 ? __builtin_bit_cast(v8h, o[TB2 + 128 + 2 * lane + 1]) : v8h{};
    };
    v8h rTBh{}, rTBl{}, rTB2ah{}, rTB2al{}, rTB2bh{}, rTB2bl{};
    if constexpr (!RELOAD) tables(ops, rTBh, rTBl, rTB2ah, rTB2al, rTB2bh, rTB2bl);
    const v16f zero16 = {};

    // output accumulators of this lane: m3 >= 0 (h = 0) or m3 < 0 (h = 1)
    float oA[L + 1], oZ[L + 1], oR[L + 1][L + 1], oP[L + 1][L + 1], oM[L + 1][L + 1];
#pragma unroll
    for (int a = 0; a <= L; ++a) {
        oA[a] = oZ[a] = 0.f;
#pragma unroll
        for (int b = 0; b <= L; ++b) oR[a][b] = oP[a][b] = oM[a][b] = 0.f;
    }

    // The node loop is software-pipelined by one stage: node k's step (A) runs
    // while node k-1's step-(D) products (issued at the end of the previous pass)
    // are still in the matrix cores; then node k-1's step (E), then node k's steps
    // (B) to (D).
    struct Front {  // node k after step (A)
        float Pc[3][L + 1], Ps[3][L + 1], dl, ep;
        const float* tb;
        int j;
    };
    struct Back {  // node k between the issue of step (D) and step (E)
        v16f sp[3];
        float d_1, d_2, e_1, e_2, a_1, a_2;
        const float* tb;
    };
    auto front1 = [&](int j) {
        Front F;
        F.j = j;
        F.tb = tab + Y.glob + j * Y.pb;
        // (A) this lane's input at node j
        coef_to_theta_fourier<L, L, true, false, true>(xr, F.tb, tab + Y.n0, BWD && h != 0, F.Pc[0], F.Ps[0], F.Pc[1], F.Ps[1],
                                          F.Pc[2], F.Ps[2], F.dl, F.ep);
        return F;
    };
    auto front2 = [&](const Front& F) {
        Back Bk;
        const float (&Pc)[3][L + 1] = F.Pc;
        const float (&Ps)[3][L + 1] = F.Ps;
        // step-(B) operands of the three polynomials of both inputs (L = 8: sin 8
        // in the sin 0 slot, cos 8 alone in a second K block)
        v8h oh[2][3], ol[2][3], oh2[3], ol2[3];
#pragma unroll
        for (int p = 0; p < 3; ++p) {
            float cv[8], sv[8];
            bool cl_[8], sl_[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                cl_[e] = e <= L;
                sl_[e] = (e >= 1 && e <= L) || (e == 0 && L >= 8);
                cv[e] = cl_[e] ? Pc[p][e] : 0.f;
                sv[e] = sl_[e] ? Ps[p][e == 0 ? (L >= 8 ? 8 : 0) : e] : 0.f;
            }
            v8h ch, cl, sh, sl;
            split8<SPLIT>(cv, cl_, neg_one, ch, cl);
            split8<SPLIT>(sv, sl_, neg_one, sh, sl);
            swap_halves(ch, sh, oh[0][p], oh[1][p]);
            if constexpr (SPLIT == 3) swap_halves(cl, sl, ol[0][p], ol[1][p]);
            if constexpr (S::KB == 2) {
                // cos 8 of the lane's own input in K element 0: kappa 16 of input 1
                // (lanes 0..31) and kappa 24 of input 2 (lanes 32..63) in one
                // operand; the tables TB2a / TB2b pick one input each
                float c8[8] = {Pc[p][L < 8 ? 0 : 8], 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
                const bool l8[8] = {true, false, false, false, false, false, false, false};
                split8<SPLIT>(c8, l8, neg_one, oh2[p], ol2[p]);
            }
        }

        // (B) fields of the six polynomials at the n_phi points
        v8h TBh = rTBh, TBl = rTBl, TB2ah = rTB2ah, TB2al = rTB2al, TB2bh = rTB2bh, TB2bl = rTB2bl;
        if constexpr (RELOAD) tables(ops + F.j * zero_i, TBh, TBl, TB2ah, TB2al, TB2bh, TB2bl);
        v16f fb[2][3];
#pragma unroll
        for (int in = 0; in < 2; ++in)
#pragma unroll
            for (int p = 0; p < 3; ++p) {
                fb[in][p] = mfma(TBh, oh[in][p], zero16);
                if constexpr (SPLIT == 3) {
                    fb[in][p] = mfma(TBh, ol[in][p], fb[in][p]);
                    fb[in][p] = mfma(TBl, oh[in][p], fb[in][p]);
                }
                if constexpr (S::KB == 2) {
                    const v8h& t2h = in ? TB2bh : TB2ah;
                    fb[in][p] = mfma(t2h, oh2[p], fb[in][p]);
                    if constexpr (SPLIT == 3) {
                        fb[in][p] = mfma(t2h, ol2[p], fb[in][p]);
                        fb[in][p] = mfma(in ? TB2bl : TB2al, oh2[p], fb[in][p]);
                    }
                }
            }

        // (C) R0 = A a + B b + C c, P1 = A b + a B, P2 = A c + a C, lane-local
        float H[3][16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            if (S::holds_point(v)) {
                const float A = fb[0][0][v], B = fb[0][1][v], C = fb[0][2][v];
                const float a = fb[1][0][v], b = fb[1][1][v], c = fb[1][2][v];
                H[0][v] = fmaf(C, c, fmaf(B, b, A * a));
                H[1][v] = fmaf(A, b, a * B);
                H[2][v] = fmaf(A, c, a * C);
            } else {
                H[0][v] = H[1][v] = H[2][v] = 0.f;
            }
        }

        // (D) spectra: R0 and P1 with table type 0, P2 with type 1
        v16f (&sp)[3] = Bk.sp;
#pragma unroll
        for (int q = 0; q < 3; ++q) {
            sp[q] = zero16;
            const int qt = q == 2 ? 1 : 0;
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                float hv[8];
                bool live[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    live[e] = 8 * b + e < 16 && S::holds_point(8 * b + e);
                    hv[e] = live[e] ? H[q][8 * b + e] : 0.f;
                }
                v8h hh, hl;
                split8<SPLIT>(hv, live, neg_one, hh, hl);
                const v4u* td = ops + 2 * (64 + (qt * NB + b) * 64 + lane);
                const v8h tdh = __builtin_bit_cast(v8h, td[0]);
                sp[q] = mfma(tdh, hh, sp[q]);
                if constexpr (SPLIT == 3) {
                    const v8h tdl = __builtin_bit_cast(v8h, td[1]);
                    sp[q] = mfma(tdh, hl, sp[q]);
                    sp[q] = mfma(tdl, hh, sp[q]);
                }
            }
        }

        bcast_halves(F.dl, Bk.d_1, Bk.d_2);
        bcast_halves(F.ep, Bk.e_1, Bk.e_2);
        bcast_halves(F.Pc[0][0], Bk.a_1, Bk.a_2);
        Bk.tb = F.tb;
        return Bk;
    };
    auto back = [&](const Back& Bk) {
        const v16f (&sp)[3] = Bk.sp;
        const float* __restrict__ tb = Bk.tb;
        const float d_1 = Bk.d_1, d_2 = Bk.d_2, e_1 = Bk.e_1, e_2 = Bk.e_2, a_1 = Bk.a_1, a_2 = Bk.a_2;
        // m3 = 0 closed forms (both halves hold the t' = 0 cosine sums)
        constexpr float NPf = static_cast<float>(S::NP);
        const float r0c0 = fmaf(-0.5f * NPf, fmaf(d_1, d_2, e_1 * e_2), sp[0][0]);
        const float sP1 = 1.41421356237309505f * sp[1][0];
        const float sP2 = 1.41421356237309505f * sp[2][0];
        const float sP4 = -NPf * fmaf(d_2, a_1, d_1 * a_2);
        const float sP3 = NPf * fmaf(e_2, a_1, e_1 * a_2);
        const float w0 = 0.5f * (sP1 + sP4), w1 = 0.5f * (sP3 + sP2);
        const float w2 = 0.5f * (sP1 - sP4), w3 = 0.5f * (sP3 - sP2);
        const float* __restrict__ m0 = tab + Y.m0;
        const float zp = fmaf(m0[0], w0, fmaf(m0[1], w1, fmaf(m0[2], w2, m0[3] * w3)));
        const float zm = fmaf(m0[4], w0, fmaf(m0[5], w1, fmaf(m0[6], w2, m0[7] * w3)));
        const float zs = h ? zm : zp;

        // (E) this node's share of the lane's outputs
#pragma unroll
        for (int l = 0; l <= L; ++l) oA[l] = fmaf(tb[Y.e0c + tri(L, 0, l)], r0c0, oA[l]);
#pragma unroll
        for (int l = 1; l <= L; ++l) oZ[l] = fmaf(tb[Y.e1z + l], zs, oZ[l]);
#pragma unroll
        for (int t = 1; t <= L; ++t) {
            const float sr = sg * sp[0][t];
            const float spp = fmaf(sg, sp[1][t], sp[2][t]);
            const float smm = fmaf(sg, sp[1][t], -sp[2][t]);
#pragma unroll
            for (int l = t; l <= L; ++l) {
                oR[t][l] = fmaf(tb[Y.e0c + tri(L, t, l)], sr, oR[t][l]);
                oP[t][l] = fmaf(tb[Y.e1p + tri(L, t, l)], spp, oP[t][l]);
                oM[t][l] = fmaf(tb[Y.e1m + tri(L, t, l)], smm, oM[t][l]);
            }
        }
    };

    // nodes j = ngrp + NG k; every wave has at least one (n_theta >= NG)
    Back prev = front2(front1(ngrp));
#pragma unroll 1
    for (int k = 1; k < S::NPW; ++k) {
        const int j = ngrp + S::NG * k;
        if (j >= S::NT) break;
        const Front F = front1(j);  // (A) of node k while (D) of node k-1 finishes
        back(prev);                 // (E) of node k-1
        prev = front2(F);           // (B) to (D) of node k
    }
    back(prev);

    // partial outputs -> LDS: node group g writes the tile at (g % 2) YB;
    // with four node groups, groups 2 and 3 write first and groups 0 and 1 add theirs
    __syncthreads();  // every wave is done with the input tiles
    // undo the input scaling: the output of a unit scales with 2^(e1 + e2)
    const int unit = 32 * T + (lane & 31);
    const int es = ex[unit] + ex[S::UNITS + unit];
    float* yr = lds + (ngrp & 1) * S::YB + unit * ST;
    if (parity) {
        // back to the parity-labelled basis (P^T, linear, so on the partial tiles):
        // (a, b) of the s = -1, +1 blocks become ((a + (-1)^l b)/sqrt2, (a - (-1)^l b)/sqrt2).
        // At m = +-t both sit in this lane (oM, oP); at m = 0 lane h = 1 holds a and
        // lane h = 0 holds b of the same unit, 32 lanes apart.
        const float hs = 0.70710678118654752440f;
#pragma unroll
        for (int t = 1; t <= L; ++t)
#pragma unroll
            for (int l = t; l <= L; ++l) {
                const float a = oM[t][l], b = (l & 1) ? -oP[t][l] : oP[t][l];
                oM[t][l] = (a + b) * hs;
                oP[t][l] = (a - b) * hs;
            }
#pragma unroll
        for (int l = 1; l <= L; ++l) {
            const float other = __shfl_xor(oZ[l], 32);
            const float a = h ? oZ[l] : other, b = (l & 1) ? -(h ? other : oZ[l]) : (h ? other : oZ[l]);
            oZ[l] = (h ? (a + b) : (a - b)) * hs;
        }
    }
    // put (ADD = false) or add (ADD = true) this lane's outputs into its row of the
    // tile; SCALED: times 2^es (with four node groups only the sum is scaled)
    auto emit = [&](auto add_tag, auto scaled_tag) {
        constexpr bool ADD = decltype(add_tag)::value;
        constexpr bool SCALED = decltype(scaled_tag)::value;
        auto put = [&](int q, float v) {
            const float w = ADD ? yr[q] + v : v;
            yr[q] = SCALED ? ldexpf(w, es) : w;
        };
        if (h == 0) {
            if constexpr (!ADD) {
                yr[0] = 0.f;        // l = 0 of s = -1
                yr[2 * BLK] = 0.f;  // l = 0 of s = +1
            }
#pragma unroll
            for (int l = 0; l <= L; ++l) put(BLK + l * l + l, oA[l]);
#pragma unroll
            for (int l = 1; l <= L; ++l) put(2 * BLK + l * l + l, oZ[l]);
        } else {
#pragma unroll
            for (int l = 1; l <= L; ++l) put(l * l + l, oZ[l]);
        }
        const int sm = h ? -1 : 1;
#pragma unroll
        for (int t = 1; t <= L; ++t)
#pragma unroll
            for (int l = t; l <= L; ++l) {
                put(BLK + l * l + l + sm * t, oR[t][l]);
                put(2 * BLK + l * l + l + sm * t, oP[t][l]);
                put(l * l + l + sm * t, oM[t][l]);
            }
    };
    if constexpr (S::NG == 2) {
        emit(std::false_type{}, std::true_type{});
    } else {
        if (ngrp >= 2) emit(std::false_type{}, std::false_type{});
        __syncthreads();
        if (ngrp < 2) emit(std::true_type{}, std::true_type{});
    }
    __syncthreads();
    store_out<NC, ST, S::UNITS, S::THREADS>(out + u0 * NC, nvalid, lds, S::YB, tid);
}

template <int L, typename TIO, int SPLIT, bool BWD>
hipError_t launch_mfma(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float* tab,
                       const uint32_t* aux, hipStream_t stream) {
    using S = MShape<L>;
    const int64_t blocks = (units + S::UNITS - 1) / S::UNITS;
    if (blocks > 0x7fffffff || aux == nullptr) return hipErrorInvalidValue;
    hipLaunchKernelGGL((spingtp_fwd_mfma_kernel<L, TIO, SPLIT, BWD>), dim3(static_cast<unsigned>(blocks)),
                       dim3(S::THREADS), 0, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                       static_cast<TIO*>(out), units, cpx2, tab, aux, -1.0f);
    return hipGetLastError();
}

struct MRegistered {
    int L, dtype;
    KernelEntry entry;
};

template <int L, typename TIO>
constexpr MRegistered reg_mfma() {
    using S = MShape<L>;
    return MRegistered{L, sizeof(TIO) == 4 ? 0 : 1,
                       KernelEntry{S::WAVES, S::UNITS, static_cast<int>(S::LDS_FLOATS * sizeof(float)), 4,
                                   &launch_mfma<L, TIO, sizeof(TIO) == 4 ? 3 : 1, false>,
                                   &launch_mfma<L, TIO, sizeof(TIO) == 4 ? 3 : 1, true>}};
}

// (at L = 4 fp32 the matrix-core kernel is 4-5 % ahead of the vector-ALU one: 0.32 vs 0.34 ns/unit)
const MRegistered kMfmaRegistry[] = {reg_mfma<4, float>(),    reg_mfma<4, uint16_t>(), reg_mfma<5, float>(),
                                     reg_mfma<5, uint16_t>(), reg_mfma<6, float>(),    reg_mfma<6, uint16_t>(),
                                     reg_mfma<7, float>(),    reg_mfma<7, uint16_t>(), reg_mfma<8, float>(),
                                     reg_mfma<8, uint16_t>()};

}  // namespace

const KernelEntry* find_mfma_kernel(int L1, int L2, int LO, int spin_mode, int dtype) {
    if (L1 != L2 || L1 != LO || spin_mode != 1) return nullptr;
    for (const MRegistered& r : kMfmaRegistry)
        if (r.L == L1 && r.dtype == dtype) return &r.entry;
    return nullptr;
}

}  // namespace spingtp
