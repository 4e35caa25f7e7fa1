// Device code of the lane-pair (L = 7, 8) and large-degree (L = 9..16) forward
// kernels shared by the translation units that instantiate them: forward.hip (the
// paper bases and the lane-pair kernel) and forward_big_parity.hip (the
// parity-basis large-degree kernels, built with another scheduling strategy).
// Everything is in an unnamed namespace: each unit keeps its own instantiations.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>
#include <utility>

#include "device_common.h"
#include "internal.h"

namespace spingtp {
namespace {

template <int L>
__device__ __forceinline__ void synth(const float (&pc)[L + 1], const float (&ps)[L + 1], const float* __restrict__ cs,
                                      const float* __restrict__ sn, float& plus, float& minus) {
    float ev = pc[0], od = 0.f;
#pragma unroll
    for (int t = 1; t <= L; ++t) {
        ev = fmaf(pc[t], cs[t], ev);
        od = fmaf(ps[t], sn[t], od);
    }
    plus = ev + od;
    minus = ev - od;
}

// Per-node spectra exchanged between the theta-node waves before the final
// projection (step E).  Slot order inside one unit's record:
//   t = 0 : R0c[0], and with spins Z+ and Z- (the m3 = 0, |s3| = 1 sums);
//   t >= 1: R0c[t], R0s[t], and with spins the four combinations
//           P1c+P2s (s3=+1, m3=+t), P1c-P2s (s3=-1, m3=+t),
//           P2c-P1s (s3=+1, m3=-t), -P2c-P1s (s3=-1, m3=-t).
// A "group" is one slot: it feeds the output coefficients l = lmin..Lout of one
// (spin block, m3).  Each group is owned by exactly one wave, which sums the
// slot over all theta nodes in a fixed order, so the result is deterministic.

template <int NG>
struct Owners {
    int owner[NG];
};

// ---------------------------------------------------------------------------
// Lane-pair kernel for L1 = L2 = Lout = L with larger L (7, 8).
//
// Lanes 2u and 2u+1 share unit u: lane 2u keeps the three polynomials of input
// 1, lane 2u+1 those of input 2 (halving the per-lane state), and each
// synthesised value is handed to the partner lane with one DPP swap.  The
// products are symmetric in the two inputs, so both lanes form them with the
// same code.  The analysis is split by trigonometric type: the even lane
// accumulates the cosine spectra of R0, P1, P2 and the odd lane the sine
// spectra, reading its own row of a cos/sin table in LDS; every other table
// value is still wave-uniform.  Step (E) pairs the output coefficient
// m3 = +t (even lane) with m3 = -t (odd lane), which use the same table entry
// (for R0 the sine table is the negated cosine table, folded into the sign of
// the exchanged value).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float swap_pair(float v) {
    // quad_perm [1,0,3,2]: exchange with the neighbouring lane
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}

template <int L, bool SPIN>
struct PairShape {
    static constexpr Layout Y = make_layout(L, L, L);
    static constexpr int NS = SPIN ? 3 : 1;
    static constexpr int NC = NS * (L + 1) * (L + 1);
    static constexpr int ST = NC | 1;
    static constexpr int NT = Y.NT;
    static constexpr int NP = Y.NP;
    static constexpr int KP = (NP - 1) / 2;
    static constexpr int UNITS = 32;
    static constexpr int WAVES = NT;
    static constexpr int THREADS = 64 * WAVES;
    // exchanged slots per unit: t = 0: (R0, unused, Z+, Z-) | t >= 1: (R0 +/-, P +/-, M +/-)
    static constexpr int T0 = SPIN ? 4 : 2;
    static constexpr int PER_T = SPIN ? 6 : 2;
    static constexpr int ND = T0 + PER_T * L;
    static constexpr int DS = ND | 1;
    static constexpr int XF = UNITS * 2 * ST;
    static constexpr int DF = NT * UNITS * DS;
    static constexpr int REGION = XF > DF ? XF : DF;
    static constexpr int TRIG = 2 * NP * (L + 1);
    static constexpr int LDS_FLOATS = REGION + UNITS * ST + TRIG;
    // pair groups: t = 0 -> R0 (l >= 0), Z (l >= 1, spins); t >= 1 -> R0, P, M (spins) or R0
    static constexpr int G0 = SPIN ? 2 : 1;
    static constexpr int GT = SPIN ? 3 : 1;
    static constexpr int NG = G0 + GT * L;
    __host__ __device__ static constexpr int t_of(int g) { return g < G0 ? 0 : 1 + (g - G0) / GT; }
    __host__ __device__ static constexpr int kind_of(int g) { return g < G0 ? (g == 0 ? 0 : 3) : (g - G0) % GT; }
    __host__ __device__ static constexpr int lmin(int g) { return kind_of(g) == 3 ? 1 : t_of(g); }
    __host__ __device__ static constexpr int size(int g) { return L + 1 - lmin(g); }
    __host__ __device__ static constexpr int slot(int g) {
        return t_of(g) == 0 ? (kind_of(g) == 0 ? 0 : 2) : T0 + PER_T * (t_of(g) - 1) + 2 * kind_of(g);
    }
};

template <int L, bool SPIN, int NW>
constexpr Owners<PairShape<L, SPIN>::NG> assign_pair_owners() {
    using P = PairShape<L, SPIN>;
    Owners<P::NG> o{};
    int load[NW] = {};
    bool done[P::NG] = {};
    for (int n = 0; n < P::NG; ++n) {
        int best = -1;
        for (int g = 0; g < P::NG; ++g)
            if (!done[g] && (best < 0 || P::size(g) > P::size(best))) best = g;
        int w = 0;
        for (int k = 1; k < NW; ++k)
            if (load[k] < load[w]) w = k;
        o.owner[best] = w;
        load[w] += P::size(best);
        done[best] = true;
    }
    return o;
}

// Steps (A)-(D) of one unit at one node for the lane pair (see above).  On
// return Q0/Q1/Q2 hold the exchanged slot values of this lane:
//   Q0[t]: R0c[t] (even lane) or -R0s[t] (odd lane), t >= 1; Q0[0] = R0c[0]
//   Q1[t]: P1c+P2s (even) or P2c-P1s (odd);  Q2[t]: P1c-P2s (even) or -P2c-P1s (odd)
//   zslot: Z+ (even lane) or Z- (odd lane), the m3 = 0, |s3| = 1 sums.
// Steps (B)-(D) from the lane's step-(A) output (theta-Fourier coefficients of its
// input at the node), over the phi-point pairs k in [k_lo, k_hi).  The spectra are
// linear in the point sums, so a node's points can be split over several waves
// whose partial spectra add up: `lead` (wave-uniform) marks the part that also
// takes the single points (phi = 0, pi) and the closed-form t = 0 terms.
template <int L, bool SPIN>
__device__ __forceinline__ void pair_spectra_from_fourier(const float (&Pc0)[L + 1], const float (&Ps0)[L + 1],
                                                          const float (&Pc1)[L + 1], const float (&Ps1)[L + 1],
                                                          const float (&Pc2)[L + 1], const float (&Ps2)[L + 1],
                                                          float dl, float ep, const float* __restrict__ g,
                                                          const float* trl, int sub, float (&Q0)[L + 1],
                                                          float (&Q1)[L + 1], float (&Q2)[L + 1], float& zslot,
                                                          int k_lo = 1, int k_hi = (make_layout(L, L, L).NP - 1) / 2 + 1,
                                                          bool lead = true) {
    constexpr Layout Y = make_layout(L, L, L);
    constexpr int TM1 = Y.TM + 1;
    constexpr int NP = Y.NP;
    const float sg = sub ? -1.f : 1.f;

    // accumulators: cosine spectra on the even lane, sine spectra on the odd lane
#pragma unroll
    for (int t = 0; t <= L; ++t) Q0[t] = Q1[t] = Q2[t] = 0.f;

    auto accumulate = [&](float vr, float v1, float v2, const float* tr) {
#pragma unroll
        for (int t = 0; t <= L; ++t) {
            const float w = tr[t];
            Q0[t] = fmaf(vr, w, Q0[t]);
            if constexpr (SPIN) {
                Q1[t] = fmaf(v1, w, Q1[t]);
                Q2[t] = fmaf(v2, w, Q2[t]);
            }
        }
    };
    // phi = 0 (and phi = pi when n_phi is even): a single point
    auto single_point = [&](int k, float sgn_t_odd) {
        float o0 = 0.f, o1 = 0.f, o2 = 0.f;
#pragma unroll
        for (int t = 0; t <= L; ++t) {
            const float c = (t & 1) ? sgn_t_odd : 1.f;
            o0 = fmaf(c, Pc0[t], o0);
            if constexpr (SPIN) o1 = fmaf(c, Pc1[t], o1), o2 = fmaf(c, Pc2[t], o2);
        }
        const float p0 = swap_pair(o0);
        float r0 = o0 * p0, q1 = 0.f, q2 = 0.f;
        if constexpr (SPIN) {
            const float p1 = swap_pair(o1), p2 = swap_pair(o2);
            r0 = fmaf(o1, p1, fmaf(o2, p2, r0));
            q1 = fmaf(o0, p1, p0 * o1);
            q2 = fmaf(o0, p2, p0 * o2);
        }
        accumulate(r0, q1, q2, trl + k * (L + 1));
    };
    if (lead) single_point(0, 1.f);
#pragma unroll 1
    for (int k = k_lo; k < k_hi; ++k) {
        const float* __restrict__ cs = g + Y.cosT + k * TM1;
        const float* __restrict__ sn = g + Y.sinT + k * TM1;
        float o0p, o0m, o1p = 0.f, o1m = 0.f, o2p = 0.f, o2m = 0.f;
        synth<L>(Pc0, Ps0, cs, sn, o0p, o0m);
        if constexpr (SPIN) {
            synth<L>(Pc1, Ps1, cs, sn, o1p, o1m);
            synth<L>(Pc2, Ps2, cs, sn, o2p, o2m);
        }
        const float p0p = swap_pair(o0p), p0m = swap_pair(o0m);
        float r0p = o0p * p0p, r0m = o0m * p0m, q1p = 0.f, q1m = 0.f, q2p = 0.f, q2m = 0.f;
        if constexpr (SPIN) {
            const float p1p = swap_pair(o1p), p1m = swap_pair(o1m);
            const float p2p = swap_pair(o2p), p2m = swap_pair(o2m);
            r0p = fmaf(o1p, p1p, fmaf(o2p, p2p, r0p));
            r0m = fmaf(o1m, p1m, fmaf(o2m, p2m, r0m));
            q1p = fmaf(o0p, p1p, p0p * o1p);
            q1m = fmaf(o0m, p1m, p0m * o1m);
            q2p = fmaf(o0p, p2p, p0p * o2p);
            q2m = fmaf(o0m, p2m, p0m * o2m);
        }
        // even lane: sums (cosine), odd lane: differences (sine)
        accumulate(fmaf(sg, r0m, r0p), fmaf(sg, q1m, q1p), fmaf(sg, q2m, q2p), trl + k * (L + 1));
    }
    if constexpr (NP % 2 == 0) {
        if (lead) single_point(NP / 2, -1.f);
    }

    // t = 0 terms (valid on the even lane, which holds input 1 and every cosine spectrum)
    zslot = 0.f;
    if constexpr (SPIN) {
        const float a0p = swap_pair(Pc0[0]);
        const float dlp = swap_pair(dl), epp = swap_pair(ep);
        if (lead) Q0[0] = fmaf(-0.5f * NP, fmaf(dl, dlp, ep * epp), Q0[0]);
        const float sP1 = 1.41421356237309505f * Q1[0];
        const float sP2 = 1.41421356237309505f * Q2[0];
        const float sP4 = lead ? -static_cast<float>(NP) * fmaf(dlp, Pc0[0], dl * a0p) : 0.f;
        const float sP3 = lead ? static_cast<float>(NP) * fmaf(epp, Pc0[0], ep * a0p) : 0.f;
        const float v0 = 0.5f * (sP1 + sP4), v1 = 0.5f * (sP3 + sP2);
        const float v2 = 0.5f * (sP1 - sP4), v3 = 0.5f * (sP3 - sP2);
        const float* m0 = g + Y.m0;
        const float zp = fmaf(m0[0], v0, fmaf(m0[1], v1, fmaf(m0[2], v2, m0[3] * v3)));
        const float zm = fmaf(m0[4], v0, fmaf(m0[5], v1, fmaf(m0[6], v2, m0[7] * v3)));
        const float zm_even = swap_pair(zm);  // all lanes active: DPP reads the even lane
        zslot = sub ? zm_even : zp;
        // cross terms: the even lane needs P2s, the odd lane P2c
#pragma unroll
        for (int t = 1; t <= L; ++t) {
            const float b = swap_pair(Q2[t]);
            const float p1 = Q1[t];
            Q1[t] = fmaf(sg, p1, b);
            Q2[t] = fmaf(sg, p1, -b);
        }
    }
#pragma unroll
    for (int t = 1; t <= L; ++t) Q0[t] *= sg;
}

template <int L, bool SPIN, bool BWD, bool PAR = false>
__device__ __forceinline__ void pair_spectra(const float* xr, const float* __restrict__ tb,
                                             const float* __restrict__ g, const float* trl, int sub,
                                             float (&Q0)[L + 1], float (&Q1)[L + 1], float (&Q2)[L + 1],
                                             float& zslot) {
    constexpr Layout Y = make_layout(L, L, L);
    float Pc0[L + 1], Ps0[L + 1], Pc1[L + 1], Ps1[L + 1], Pc2[L + 1], Ps2[L + 1], dl, ep;
    coef_to_theta_fourier<L, L, SPIN, PAR>(xr, tb, g + Y.n0, BWD && sub != 0, Pc0, Ps0, Pc1, Ps1, Pc2, Ps2, dl, ep);
    pair_spectra_from_fourier<L, SPIN>(Pc0, Ps0, Pc1, Ps1, Pc2, Ps2, dl, ep, g, trl, sub, Q0, Q1, Q2, zslot);
}

// Step (A) a few degrees at a time.  The large-degree kernel stages slots
// LA^2 .. LB^2 - 1 of every spin block of its input rows in LDS (one chunk of
// degrees l in [LA, LB)) and adds each chunk's terms to sums that persist across
// the chunks.  Every sum still runs over l in increasing order, so the results
// are those of coef_to_theta_fourier.
template <int L, bool SPIN>
struct ThetaSums {
    float sc[L + 1], ss[L + 1];                        // spin 0: cosine, sine (t >= 1)
    float up[L + 1], vp[L + 1], um[L + 1], vm[L + 1];  // |s| = 1, t >= 1
    float wpl, wmi;                                    // |s| = 1, t = 0
};

template <int L, bool SPIN>
__device__ __forceinline__ void theta_sums_zero(ThetaSums<L, SPIN>& a) {
#pragma unroll
    for (int t = 0; t <= L; ++t) a.sc[t] = a.ss[t] = a.up[t] = a.vp[t] = a.um[t] = a.vm[t] = 0.f;
    a.wpl = a.wmi = 0.f;
}

// s: the lane's staged row, block b (spins -1, 0, +1, or 0 alone) at s + b CW with
// CW = LB^2 - LA^2 slots, slot q of a block at offset q - LA^2.
template <int L, bool SPIN, bool PAR, int LA, int LB>
__device__ __forceinline__ void theta_sums_add(const float* s, const float* __restrict__ tb, ThetaSums<L, SPIN>& a) {
    constexpr Layout Y = make_layout(L, 0, 0);
    constexpr int CW = LB * LB - LA * LA, O = LA * LA;
    const float* x0 = s + (SPIN ? CW : 0);
    // (scheduling fences per order t keep one order's row values in flight at a time)
#pragma unroll
    for (int t = 0; t < LB; ++t) {
#pragma unroll
        for (int l = (t > LA ? t : LA); l < LB; ++l) {
            a.sc[t] = fmaf(x0[l * l + l + t - O], tb[Y.a0c + tri(L, t, l)], a.sc[t]);
            if (t > 0) a.ss[t] = fmaf(x0[l * l + l - t - O], tb[Y.a0s + tri(L, t, l)], a.ss[t]);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (SPIN) {
        const float* xm = s;
        const float* xp = s + 2 * CW;
        // paper-basis -1 and +1 values of slot q from the parity-labelled ones (up to
        // the factor 1/sqrt2 applied to the finished sums)
        auto vm_of = [&](int q) { return PAR ? xm[q - O] + xp[q - O] : xm[q - O]; };
        auto vp_of = [&](int q, int l) {
            return PAR ? ((l & 1) ? xp[q - O] - xm[q - O] : xm[q - O] - xp[q - O]) : xp[q - O];
        };
#pragma unroll
        for (int t = 1; t < LB; ++t) {
#pragma unroll
            for (int l = (t > LA ? t : LA); l < LB; ++l) {
                const float wp = tb[Y.aup + tri(L, t, l)];
                const float wm = tb[Y.aum + tri(L, t, l)];
                a.up[t] = fmaf(vp_of(l * l + l + t, l), wp, a.up[t]);
                a.vp[t] = fmaf(vp_of(l * l + l - t, l), wp, a.vp[t]);
                a.um[t] = fmaf(vm_of(l * l + l + t), wm, a.um[t]);
                a.vm[t] = fmaf(vm_of(l * l + l - t), wm, a.vm[t]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int l = (LA > 1 ? LA : 1); l < LB; ++l) {
            const float w = tb[Y.aw + l];
            a.wpl = fmaf(vp_of(l * l + l, l), w, a.wpl);
            a.wmi = fmaf(vm_of(l * l + l), w, a.wmi);
        }
    }
}

// The step-(A) outputs from the finished sums (the closing steps of coef_to_theta_fourier).
template <int L, bool SPIN, bool PAR>
__device__ __forceinline__ void theta_sums_finish(const ThetaSums<L, SPIN>& a, const float* __restrict__ n0,
                                                  bool second, float (&Ac)[L + 1], float (&As)[L + 1],
                                                  float (&Bc)[L + 1], float (&Bs)[L + 1], float (&Cc)[L + 1],
                                                  float (&Cs)[L + 1], float& dl, float& ep) {
#pragma unroll
    for (int t = 0; t <= L; ++t) {
        Ac[t] = a.sc[t];
        As[t] = t > 0 ? a.ss[t] : 0.f;
    }
    if constexpr (SPIN) {
        const float hs = PAR ? 0.70710678118654752440f : 1.f;
#pragma unroll
        for (int t = 1; t <= L; ++t) {
            float up = a.up[t], vp = a.vp[t], um = a.um[t], vm = a.vm[t];
            if constexpr (PAR) up *= hs, vp *= hs, um *= hs, vm *= hs;
            Bc[t] = up + um;
            Bs[t] = -(vp + vm);
            Cc[t] = vp - vm;
            Cs[t] = up - um;
        }
        float wpl = a.wpl, wmi = a.wmi;
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

// Writes one unit's slot record (layout of PairShape) for this lane.
template <int L, bool SPIN>
__device__ __forceinline__ void pair_publish(float* D, int sub, const float (&Q0)[L + 1], const float (&Q1)[L + 1],
                                             const float (&Q2)[L + 1], float zslot) {
    constexpr int T0 = SPIN ? 4 : 2, PER_T = SPIN ? 6 : 2;
    D[sub] = Q0[0];
    if constexpr (SPIN) D[2 + sub] = zslot;
#pragma unroll
    for (int t = 1; t <= L; ++t) {
        float* d = D + T0 + PER_T * (t - 1);
        d[sub] = Q0[t];
        if constexpr (SPIN) {
            d[2 + sub] = Q1[t];
            d[4 + sub] = Q2[t];
        }
    }
}

// ---------------------------------------------------------------------------
// Large-degree kernel (L = 9..16, fp32 or bf16 I/O, fp32 arithmetic).  More nodes than a workgroup has
// waves, and 32-unit input tiles that no longer fit in LDS: the nodes are
// processed in rounds of W waves.  In each round the workgroup stages the tile's
// input rows in LDS a chunk of degrees at a time (coalesced loads, the next
// chunk's loads in flight while the waves work on the current one) and every
// lane pair runs step (A) for its wave's node from there; the spectra of the
// round are then exchanged in LDS (the same region), and every output group's
// owner lane accumulates the round's contribution into the output row (written
// in round 0, then read, added and written by the same lane in later rounds:
// ordered, deterministic).  The output rows of the tile live in LDS across the
// rounds and leave in one coalesced store.
// ---------------------------------------------------------------------------
template <int L, bool SPIN, int W>
struct BigShape {
    using PS = PairShape<L, SPIN>;
    static constexpr Layout Y = make_layout(L, L, L);
    static constexpr int NC = PS::NC;
    static constexpr int NT = Y.NT;
    static constexpr int NP = Y.NP;
    static constexpr int UNITS = 32;
    static constexpr int WAVES = W;
    static constexpr int THREADS = 64 * W;
    static constexpr int ROUNDS = (NT + W - 1) / W;
    static constexpr int TRIG = 2 * NP * (L + 1);
    static constexpr int STO = NC | 1;  // odd row stride of the output tile
    // A round's spectra go through LDS in K parts, part k holding the slots of the
    // orders t in [tlo(k), tlo(k + 1)); K is the fewest parts (up to 4) with which
    // the output tile stays in LDS next to one part of W waves' spectra.
    __host__ __device__ static constexpr int tlo(int k, int K) { return k * (L + 1) / K; }
    __host__ __device__ static constexpr int sbase(int t) { return t == 0 ? 0 : PS::T0 + PS::PER_T * (t - 1); }
    __host__ __device__ static constexpr int pwidth(int K) {
        int w = 0;
        for (int k = 0; k < K; ++k) {
            const int a = sbase(tlo(k, K)), b = tlo(k + 1, K) > L ? PS::ND : sbase(tlo(k + 1, K));
            w = b - a > w ? b - a : w;
        }
        return w | 1;
    }
    __host__ __device__ static constexpr bool fits(int K) {
        return (W * UNITS * pwidth(K) + TRIG + UNITS * STO) * 4 <= 160 * 1024;
    }
    static constexpr int K = fits(1) ? 1 : fits(2) ? 2 : fits(3) ? 3 : fits(4) ? 4 : 1;
    static constexpr bool OUT_LDS = fits(K);
    static constexpr int DSP = pwidth(K);  // record stride of one part
    static constexpr int DF = W * UNITS * DSP;
    static constexpr int LDS_FLOATS = DF + TRIG + (OUT_LDS ? UNITS * STO : 0);
    __host__ __device__ static constexpr int part_of_t(int t) {
        int k = 0;
        while (k + 1 < K && t >= tlo(k + 1, K)) ++k;
        return k;
    }
    // Step (A) reads the tile's 64 input rows (two per unit: lane 2u + i holds input
    // i + 1 of unit u) from LDS.  They are staged in the spectra region, which is
    // free until the round's spectra are published, one chunk of degrees
    // [chunk_lo(c), chunk_lo(c + 1)) at a time: NS blocks of at most SCAP slots per
    // row, odd row stride.
    static constexpr int NS = SPIN ? 3 : 1;
    static constexpr int BB = (L + 1) * (L + 1);
    static constexpr int SROW = (DF / 64) % 2 ? DF / 64 : DF / 64 - 1;
    static constexpr int SCAP = SROW / NS;
    static_assert(2 * L + 1 <= SCAP, "a chunk holds at least one degree");
    __host__ __device__ static constexpr int chunk_end(int la) {  // as many degrees as fit
        int lb = la + 1;
        while (lb <= L && (lb + 1) * (lb + 1) - la * la <= SCAP) ++lb;
        return lb;
    }
    __host__ __device__ static constexpr int chunk_lo(int c) {
        int la = 0;
        for (int i = 0; i < c; ++i) la = chunk_end(la);
        return la;
    }
    __host__ __device__ static constexpr int n_chunks() {
        int n = 0;
        for (int la = 0; la <= L; la = chunk_end(la)) ++n;
        return n;
    }
    static constexpr int NCH = n_chunks();
};

template <typename F, int... I>
__device__ __forceinline__ void for_each_index(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}

// Owners of the output groups with several spectrum parts: each part's groups are
// spread over the waves by size (largest first, least-loaded wave).
template <int L, bool SPIN, int NW, int K>
constexpr Owners<PairShape<L, SPIN>::NG> assign_part_owners() {
    using P = PairShape<L, SPIN>;
    using B = BigShape<L, SPIN, NW>;
    Owners<P::NG> o{};
    for (int k = 0; k < K; ++k) {
        int load[NW] = {};
        bool done[P::NG] = {};
        for (;;) {
            int best = -1;
            for (int g = 0; g < P::NG; ++g)
                if (!done[g] && B::part_of_t(P::t_of(g)) == k && (best < 0 || P::size(g) > P::size(best))) best = g;
            if (best < 0) break;
            int w = 0;
            for (int q = 1; q < NW; ++q)
                if (load[q] < load[w]) w = q;
            o.owner[best] = w;
            load[w] += P::size(best);
            done[best] = true;
        }
    }
    return o;
}

// pair_publish restricted to the orders t in [T_LO, T_HI), slot s stored at s - sbase(T_LO).
template <int L, bool SPIN, int T_LO, int T_HI>
__device__ __forceinline__ void pair_publish_part(float* D, int sub, const float (&Q0)[L + 1],
                                                  const float (&Q1)[L + 1], const float (&Q2)[L + 1], float zslot) {
    constexpr int T0 = SPIN ? 4 : 2, PER_T = SPIN ? 6 : 2;
    constexpr int base = T_LO == 0 ? 0 : T0 + PER_T * (T_LO - 1);
    if constexpr (T_LO == 0) {
        D[sub] = Q0[0];
        if constexpr (SPIN) D[2 + sub] = zslot;
    }
#pragma unroll
    for (int t = (T_LO > 1 ? T_LO : 1); t < T_HI; ++t) {
        float* d = D + T0 + PER_T * (t - 1) - base;
        d[sub] = Q0[t];
        if constexpr (SPIN) {
            d[2 + sub] = Q1[t];
            d[4 + sub] = Q2[t];
        }
    }
}

// Whether the last round splits its nodes' phi points over the idle waves.  Measured
// on 262,144 units: it pays wherever the last round leaves waves idle, except where
// the extra per-round state costs spills (paper basis L = 9: 0.89 -> 0.96 ms;
// parity basis L = 12: 2.67 -> 2.93 ms; the scalar-spin kernels up to L = 13).
template <int L, bool SPIN, bool PAR>
constexpr bool big_split_last() {
    if (!SPIN) return L == 16;
    if (PAR) return L == 11 || L == 13 || L == 14 || L == 16;
    return L >= 11;
}

// Whether the staging loads may stay hoisted out of the round loop: the compiler then
// loads every chunk's rows once per tile and keeps them in registers, which pays
// where they fit without spilling (L = 9 0.88 against 1.01 ms, L = 12 2.61 against
// 2.80 on 262,144 units; from L = 13 on they spill 22-61 VGPRs, and the scalar-spin
// kernels gain nothing).
template <int L, bool SPIN, bool PAR>
constexpr bool big_hoist_rows() {
    return SPIN && L <= 12;
}

// PAR (spins only): the plan's basis is the parity-labelled one; a separate
// instantiation, since a run-time switch between the two step-(A) forms costs the
// paper-basis kernels registers.
// zero: 0 from the launcher.  The input rows are the same in every round, so the
// compiler hoists the staging loads of all chunks out of the round loop; where they
// do not fit in registers it holds them in scratch (106 spilled VGPRs at L = 16).
// Offsetting them by round * zero keeps them in the loop, in flight one chunk ahead
// (big_hoist_rows picks the degrees where the hoisted form fits).
// TIO: float (fp32 I/O) or uint16_t (bf16 I/O: rows widened to fp32 as they are staged,
// the output tile rounded to nearest even as it is stored; all arithmetic in fp32).
// PAD: a plan with mixed degrees (L1, L2, Lout), all <= L, read from deg (ignored
// otherwise).  Such a product equals the degree-L one of the same functions (x1, x2
// padded with zeros above their degrees) truncated to Lout, since the degree-L grid is
// exact for the products of degree <= 3 L >= L1 + L2 + Lout: the rows are staged with
// zeros above L1 and L2 and the output tile is stored up to Lout.  A separate
// instantiation: the run-time row strides and bounds cost the equal-degree kernels
// registers (L = 16: 2 -> 147 spilled VGPRs).
template <int L, bool SPIN, int W, bool BWD, bool PAR, typename TIO, bool PAD>
__global__ __launch_bounds__((BigShape<L, SPIN, W>::THREADS)) void spingtp_fwd_big_kernel(
    const TIO* __restrict__ x1, const TIO* __restrict__ x2, TIO* __restrict__ out, int64_t units, int64_t cpx2,
    const float* __restrict__ tab, const uint32_t* __restrict__ deg, int zero) {
    using B = BigShape<L, SPIN, W>;
    constexpr bool F32 = std::is_same<TIO, float>::value;
    static_assert(F32 || B::OUT_LDS, "bf16 I/O needs the output tile in LDS");
    static_assert(!PAD || B::OUT_LDS, "mixed degrees need the output tile in LDS");
    using P = typename B::PS;
    constexpr Layout Y = B::Y;
    constexpr bool SPLIT = big_split_last<L, SPIN, PAR>();
    constexpr int TM1 = Y.TM + 1;
    constexpr int BO = (L + 1) * (L + 1);
    __shared__ float lds[B::LDS_FLOATS];
    float* D = lds;
    float* TR = lds + B::DF;
    float* YT = TR + B::TRIG;  // output tile (OUT_LDS only)

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int u = lane >> 1;
    const int sub = lane & 1;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t u0 = static_cast<int64_t>(blockIdx.x) * B::UNITS;
    const int nvalid = static_cast<int>(units - u0 < B::UNITS ? units - u0 : B::UNITS);
    const bool valid = u < nvalid;
    const int64_t row = u0 + (valid ? u : 0);  // invalid lanes compute on a valid row, store nothing
    const float* g = tab;
    // slots per spin block of the x1, x2 and output rows (their degrees' (l + 1)^2)
    const int bb1 = PAD ? static_cast<int>((deg[0] + 1) * (deg[0] + 1)) : B::BB;
    const int bb2 = PAD ? static_cast<int>((deg[1] + 1) * (deg[1] + 1)) : B::BB;
    const int bbo = PAD ? static_cast<int>((deg[2] + 1) * (deg[2] + 1)) : B::BB;
    float* orow = nullptr;  // the output row in global memory (fp32 without the LDS tile)
    if constexpr (F32) orow = out + row * B::NC;
    // staging: TPR threads per input row (row r = lane r of every wave)
    constexpr int TPR = B::THREADS / 64;
    static_assert(B::THREADS % 64 == 0, "whole waves");
    const int sr = tid / TPR, sk = tid % TPR;
    const int64_t srow = u0 + ((sr >> 1) < nvalid ? (sr >> 1) : 0);
    const int sbb = (sr & 1) ? bb2 : bb1;  // this thread's row: slots per spin block
    const TIO* ssrc;
    if constexpr (PAD) ssrc = (sr & 1) ? x2 + (srow / cpx2) * (B::NS * bb2) : x1 + srow * (B::NS * bb1);
    else ssrc = (sr & 1) ? x2 + (srow / cpx2) * B::NC : x1 + srow * B::NC;

    for (int i = tid; i < B::TRIG; i += B::THREADS) {
        const int sb = i / (B::NP * (L + 1));
        const int r = i - sb * (B::NP * (L + 1));
        const int k = r / (L + 1), t = r - k * (L + 1);
        TR[i] = g[(sb ? Y.sinT : Y.cosT) + k * TM1 + t];
    }
    // parity basis: the |s| = 1 blocks of each input row are mixed by P as step (A)
    // reads them, and the finished output rows by P^T before they are final
    static_assert(SPIN || !PAR, "the parity basis only mixes |s| = 1 blocks");
    if constexpr (SPIN) {  // l = 0 slots of the |s| = 1 blocks
        if constexpr (B::OUT_LDS) {
            if (wave == 0) YT[u * B::STO + (sub ? 2 * BO : 0)] = 0.f;
        } else {
            if (wave == 0 && valid) orow[sub ? 2 * BO : 0] = 0.f;
        }
    }
    __syncthreads();

    constexpr int K = B::K;
    constexpr Owners<P::NG> own = K == 1 ? assign_pair_owners<L, SPIN, W>() : assign_part_owners<L, SPIN, W, K>();
#pragma unroll 1
    for (int r = 0; r < B::ROUNDS; ++r) {
        // A round takes nr nodes.  With SPLIT, a round with fewer nodes than waves (the
        // last one) splits each node's phi points over nsplit = W / nr waves: wave w
        // takes node r W + w % nr, part w / nr, and publishes a partial record; the
        // owners' sum over the nw = nr nsplit records below adds the parts up.
        const int nr = (B::NT - r * W) < W ? (B::NT - r * W) : W;
        const int nsplit = SPLIT ? W / nr : 1, nw = SPLIT ? nr * nsplit : nr;
        const int node = SPLIT ? r * W + wave % nr : r * W + wave;
        const int ppart = SPLIT ? wave / nr : 0;
        const bool active = SPLIT ? wave < nw : node < B::NT;
        float Q0[L + 1], Q1[L + 1], Q2[L + 1], zslot;
        // (A) chunk by chunk: stage the 64 rows' slots of the chunk's degrees, then
        // every wave adds them to its node's sums
        const float* tb = tab + Y.glob + (active ? node : 0) * Y.pb;
        ThetaSums<L, SPIN> acc;
        theta_sums_zero(acc);
        // software pipeline: chunk c + 1's global loads are in flight while the
        // waves work on chunk c
        constexpr int IT = (B::SCAP + TPR - 1) / TPR;  // staged values per block and thread
        float pre[B::NS][IT];
        const TIO* rsrc = big_hoist_rows<L, SPIN, PAR>() ? ssrc : ssrc + r * zero;
        auto widen = [](TIO v) {
            if constexpr (F32) return v;
            else return __uint_as_float(static_cast<uint32_t>(v) << 16);
        };
        auto fetch = [&](auto cc) {
            constexpr int c = decltype(cc)::value;
            constexpr int LA = B::chunk_lo(c), LB = B::chunk_lo(c + 1);
            constexpr int CW = LB * LB - LA * LA;
#pragma unroll
            for (int b = 0; b < B::NS; ++b)
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int q = sk + it * TPR;
                    if (it * TPR >= CW) continue;
                    if constexpr (PAD)
                        pre[b][it] = (q < CW && LA * LA + q < sbb) ? widen(rsrc[b * sbb + LA * LA + q]) : 0.f;
                    else
                        pre[b][it] = q < CW ? widen(rsrc[b * B::BB + LA * LA + q]) : 0.f;
                }
        };
        auto chunk = [&](auto cc) {
            constexpr int c = decltype(cc)::value;
            constexpr int LA = B::chunk_lo(c), LB = B::chunk_lo(c + 1);
            constexpr int CW = LB * LB - LA * LA, STR = (B::NS * CW) | 1;
            if constexpr (c > 0) __syncthreads();  // every wave is done with the previous chunk
#pragma unroll
            for (int b = 0; b < B::NS; ++b)
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int q = sk + it * TPR;
                    if (it * TPR < CW && q < CW) D[sr * STR + b * CW + q] = pre[b][it];
                }
            __syncthreads();
            if constexpr (c + 1 < B::NCH) fetch(std::integral_constant<int, c + 1>{});
            if (active) theta_sums_add<L, SPIN, PAR, LA, LB>(D + lane * STR, tb, acc);
        };
        fetch(std::integral_constant<int, 0>{});
        for_each_index(chunk, std::make_integer_sequence<int, B::NCH>{});
        __syncthreads();  // the staged rows are read before the spectra take the region
        if (active) {
            float Pc0[L + 1], Ps0[L + 1], Pc1[L + 1], Ps1[L + 1], Pc2[L + 1], Ps2[L + 1], dl, ep;
            theta_sums_finish<L, SPIN, PAR>(acc, g + Y.n0, BWD && sub != 0, Pc0, Ps0, Pc1, Ps1, Pc2, Ps2, dl, ep);
            const float* trl = TR + sub * (B::NP * (L + 1));
            if constexpr (SPLIT) {
                constexpr int KP = (B::NP - 1) / 2;  // phi-point pairs k = 1..KP
                const int k_lo = 1 + ppart * KP / nsplit, k_hi = 1 + (ppart + 1) * KP / nsplit;
                pair_spectra_from_fourier<L, SPIN>(Pc0, Ps0, Pc1, Ps1, Pc2, Ps2, dl, ep, g, trl, sub, Q0, Q1, Q2,
                                                   zslot, k_lo, k_hi, ppart == 0);
            } else {
                pair_spectra_from_fourier<L, SPIN>(Pc0, Ps0, Pc1, Ps1, Pc2, Ps2, dl, ep, g, trl, sub, Q0, Q1, Q2,
                                                   zslot);
            }
        }
        // the round's spectra in K parts (orders t in [tlo(k), tlo(k + 1))): publish
        // part k, then every owner of a group of part k adds the round's nodes
        auto part = [&](auto kc) {
            constexpr int k = decltype(kc)::value;
            constexpr int T_LO = B::tlo(k, K), T_HI = B::tlo(k + 1, K);
            if (active)
                pair_publish_part<L, SPIN, T_LO, T_HI>(D + (wave * B::UNITS + u) * B::DSP, sub, Q0, Q1, Q2, zslot);
            __syncthreads();
#pragma unroll
            for (int gi = 0; gi < P::NG; ++gi) {
                if (B::part_of_t(P::t_of(gi)) != k || own.owner[gi] != wave) continue;
                const int t = P::t_of(gi), kind = P::kind_of(gi);
                int tab_base = Y.e0c, blk = SPIN ? BO : 0;
                if (kind == 1) tab_base = Y.e1p, blk = 2 * BO;
                if (kind == 2) tab_base = Y.e1m, blk = 0;
                if (kind == 3) tab_base = Y.e1z, blk = sub ? 0 : 2 * BO;
                float acc[L + 1];
#pragma unroll
                for (int l = 0; l <= L; ++l) acc[l] = 0.f;
#pragma unroll 1
                for (int jj = 0; jj < nw; ++jj) {
                    const float d = D[(jj * B::UNITS + u) * B::DSP + P::slot(gi) - B::sbase(T_LO) + sub];
                    const float* te = tab + Y.glob + (r * W + (SPLIT ? jj % nr : jj)) * Y.pb;
#pragma unroll
                    for (int l = P::lmin(gi); l <= L; ++l)
                        acc[l] = fmaf(te[kind == 3 ? tab_base + l : tab_base + tri(L, t, l)], d, acc[l]);
                }
                if (valid && !(t == 0 && kind == 0 && sub)) {
                    float* yrow = B::OUT_LDS ? YT + u * B::STO : orow;
#pragma unroll
                    for (int l = P::lmin(gi); l <= L; ++l) {
                        float* o = yrow + blk + l * l + l + (sub ? -t : t);
                        *o = (r == 0) ? acc[l] : *o + acc[l];
                    }
                }
            }
            __syncthreads();
        };
        part(std::integral_constant<int, 0>{});
        if constexpr (K > 1) part(std::integral_constant<int, 1>{});
        if constexpr (K > 2) part(std::integral_constant<int, 2>{});
        if constexpr (K > 3) part(std::integral_constant<int, 3>{});
    }
    if constexpr (B::OUT_LDS) {
        if constexpr (PAR) {
            parity_mix_rows<L>(YT, B::STO, nvalid, true, tid, B::THREADS);
            __syncthreads();
        }
        if constexpr (!PAD) {
            store_tile<B::NC, B::STO>(out + u0 * B::NC, nvalid, YT, tid, B::THREADS);
        } else {  // slots of degree <= Lout of each spin block
            const int nco = B::NS * bbo;
            for (int i = tid; i < nvalid * nco; i += B::THREADS) {
                const int uu = i / nco, rem = i - uu * nco, b = rem / bbo, q = rem - b * bbo;
                const float v = YT[uu * B::STO + b * B::BB + q];
                if constexpr (F32) out[(u0 + uu) * nco + rem] = v;
                else out[(u0 + uu) * nco + rem] = f32_to_bf16(v);
            }
        }
    } else if constexpr (PAR && F32) {
        // the rows were accumulated in global memory by several waves; the barrier
        // that ends the last round orders those stores before these reads
        parity_mix_rows<L>(out + u0 * B::NC, B::NC, nvalid, true, tid, B::THREADS);
    }
}

// deg: the three degrees for PAD (launches of the mixed-degree plans), else unused.
template <int L, bool SPIN, int W, bool BWD, bool PAR, typename TIO = float, bool PAD = false>
hipError_t launch_big(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float* tab,
                      const uint32_t* deg, hipStream_t stream) {
    using B = BigShape<L, SPIN, W>;
    const int64_t blocks = (units + B::UNITS - 1) / B::UNITS;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    if (PAD && deg == nullptr) return hipErrorInvalidValue;
    hipLaunchKernelGGL((spingtp_fwd_big_kernel<L, SPIN, W, BWD, PAR, TIO, PAD>), dim3(static_cast<unsigned>(blocks)),
                       dim3(B::THREADS), 0, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                       static_cast<TIO*>(out), units, cpx2, tab, PAD ? deg : nullptr, 0);
    return hipGetLastError();
}

// Nodes per round: eight waves (two per SIMD at up to 256 VGPRs); the spectra go
// through LDS in as many parts as the output tile needs to stay there (BigShape::K).
template <int L, bool SPIN>
constexpr int big_waves() {
    return 8;
}

}  // namespace
}  // namespace spingtp
