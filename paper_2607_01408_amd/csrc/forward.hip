// Fused SpinGTP forward kernel for gfx950 (CDNA4) and its launch entry point.
//
// Method (paper App. B proof of the runtime proposition; Sec. 3.2 eq.
// generalized_gaunt): each output coefficient is the projection of the
// pointwise product of the two input fields, so a unit is
//   (A) coefficients -> theta-Fourier form of the fields at a Gauss-Legendre node
//   (B) synthesis of the fields at the n_phi uniform phi nodes
//   (C) spin-pair products  h_s3 = sum_{s1+s2=s3} f1_s1 f2_s2
//   (D) analysis of the products onto cos/sin(t phi)
//   (E) projection onto the output coefficients with the node's weight,
// summed over the n_theta nodes.  The grid is exact (layout.h), so the result
// equals the Gaunt contraction up to fp32 rounding.
//
// Work mapping.  A workgroup owns 64 units (one per lane) and one wave per
// theta node, so every table value a wave reads is the same for its 64 lanes
// and comes from the scalar cache; the per-unit data lives in VGPRs.  The two
// input tiles are staged through LDS with coalesced 16-byte loads; the partial
// outputs of the theta-node waves are summed in LDS with ds_add_f32 and written
// back with coalesced 16-byte stores.  Fields, products and spectra never leave
// the CU.
//
// Spin structure for spins {-1, 0, +1} (real basis, eq. real_swsh / App. C):
// for t = |m| >= 1 the field of spin -1 is the complex conjugate of the field of
// spin +1, so each input carries three real trigonometric polynomials per node:
//   A = f_0,   B~ = sqrt2 (Re f+ + Re f-)/2,   C~ = sqrt2 (Im f+ - Im f-)/2,
// plus two m = 0 constants delta = Re(f- - conj f+), eps = Im(f- - conj f+).
// The only output combinations the real projection needs are
//   R0 = Re h_0 = A a + B~ b~ + C~ c~ - (d1 d2 + e1 e2)/2,
//   P1 = Re h+ + Re h- = sqrt2 (A b~ + a B~),   P2 = Im h+ - Im h- = sqrt2 (A c~ + a C~),
// and, at m3 = 0 only, Re h+ - Re h- and Im h+ + Im h-, which follow from the
// t = 0 coefficients and delta, eps in closed form.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.h"
#include "forward_pair.h"
#include "internal.h"

namespace spingtp {
namespace {

template <int LO, bool SPIN>
struct Spectra {
    static constexpr int PER_T = SPIN ? 6 : 2;
    static constexpr int ND = (SPIN ? 3 : 1) + PER_T * LO;  // slots per unit per node
    static constexpr int DS = ND | 1;                        // odd LDS stride
    static constexpr int NG = ND;                            // one group per slot
    __host__ __device__ static constexpr int t_of(int g) { return g < (SPIN ? 3 : 1) ? 0 : 1 + (g - (SPIN ? 3 : 1)) / PER_T; }
    __host__ __device__ static constexpr int slot_of(int g) { return g < (SPIN ? 3 : 1) ? g : (g - (SPIN ? 3 : 1)) % PER_T; }
    __host__ __device__ static constexpr int lmin(int g) {
        return t_of(g) == 0 ? (slot_of(g) == 0 ? 0 : 1) : t_of(g);
    }
    __host__ __device__ static constexpr int size(int g) { return LO + 1 - lmin(g); }
};


// Longest-processing-time assignment of the groups to NW waves.
template <int LO, bool SPIN, int NW>
constexpr Owners<Spectra<LO, SPIN>::NG> assign_owners() {
    using SP = Spectra<LO, SPIN>;
    Owners<SP::NG> o{};
    int load[NW] = {};
    bool done[SP::NG] = {};
    for (int n = 0; n < SP::NG; ++n) {
        int best = -1;
        for (int g = 0; g < SP::NG; ++g)
            if (!done[g] && (best < 0 || SP::size(g) > SP::size(best))) best = g;
        int w = 0;
        for (int k = 1; k < NW; ++k)
            if (load[k] < load[w]) w = k;
        o.owner[best] = w;
        load[w] += SP::size(best);
        done[best] = true;
    }
    return o;
}

template <int L1, int L2, int LO, bool SPIN>
struct Shape {
    static constexpr Layout Y = make_layout(L1, L2, LO);
    static constexpr int NS = SPIN ? 3 : 1;
    static constexpr int NC1 = NS * (L1 + 1) * (L1 + 1);
    static constexpr int NC2 = NS * (L2 + 1) * (L2 + 1);
    static constexpr int NCO = NS * (LO + 1) * (LO + 1);
    static constexpr int ST1 = NC1 | 1;  // odd strides: conflict-free ds_read_b32 across lanes
    static constexpr int ST2 = NC2 | 1;
    static constexpr int STO = NCO | 1;
    static constexpr int NT = Y.NT;
    static constexpr int NP = Y.NP;
    static constexpr int KP = (NP - 1) / 2;
    static constexpr int WAVES = NT;
    static constexpr int THREADS = 64 * WAVES;
    // LDS: the input tiles, later reused for the per-node spectra, then the output tile
    static constexpr int XF = 64 * (ST1 + ST2);
    static constexpr int DF = NT * 64 * Spectra<LO, SPIN>::DS;
    static constexpr int REGION = XF > DF ? XF : DF;
    static constexpr int LDS_FLOATS = REGION + 64 * STO;
};

template <int L1, int L2, int LO, bool SPIN, typename TIO>
__global__ __launch_bounds__((Shape<L1, L2, LO, SPIN>::THREADS)) void spingtp_fwd_kernel(
    const TIO* __restrict__ x1, const TIO* __restrict__ x2, TIO* __restrict__ out, int64_t units, int64_t cpx2,
    const float* __restrict__ tab) {
    using S = Shape<L1, L2, LO, SPIN>;
    constexpr Layout Y = S::Y;
    constexpr int LA = Y.LA;
    constexpr int TM1 = Y.TM + 1;
    __shared__ float lds[S::LDS_FLOATS];
    float* X1 = lds;
    float* X2 = X1 + 64 * S::ST1;
    float* YT = lds + S::REGION;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int node = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t u0 = static_cast<int64_t>(blockIdx.x) * 64;
    const int nvalid = static_cast<int>(units - u0 < 64 ? units - u0 : 64);

    for (int i = tid; i < 64 * S::STO; i += S::THREADS) YT[i] = 0.f;
    load_tile<S::NC1, S::ST1>(x1 + u0 * S::NC1, nvalid, X1, tid, S::THREADS);
    if (cpx2 == 1)
        load_tile<S::NC2, S::ST2>(x2 + u0 * S::NC2, nvalid, X2, tid, S::THREADS);
    else
        load_tile_shared<S::NC2, S::ST2>(x2, u0, nvalid, cpx2, X2, tid, S::THREADS);
    __syncthreads();
    bool parity = false;  // uniform
    if constexpr (SPIN) {
        parity = tab[Y.par] != 0.f;
        if (parity) {
            parity_mix_rows<L1>(X1, S::ST1, nvalid, false, tid, S::THREADS);
            parity_mix_rows<L2>(X2, S::ST2, nvalid, false, tid, S::THREADS);
            __syncthreads();
        }
    }

    const float* __restrict__ g = tab;
    const float* __restrict__ tb = tab + Y.glob + node * Y.pb;

    // (A) both inputs at this node
    float Ac[L1 + 1], As[L1 + 1], Bc[L1 + 1], Bs[L1 + 1], Cc[L1 + 1], Cs[L1 + 1], d1, e1;
    float ac[L2 + 1], as[L2 + 1], bc[L2 + 1], bs[L2 + 1], cc[L2 + 1], cs2[L2 + 1], d2, e2;
    coef_to_theta_fourier<L1, LA, SPIN>(X1 + lane * S::ST1, tb, g + Y.n0, false, Ac, As, Bc, Bs, Cc, Cs, d1, e1);
    coef_to_theta_fourier<L2, LA, SPIN>(X2 + lane * S::ST2, tb, g + Y.n0, true, ac, as, bc, bs, cc, cs2, d2, e2);

    // (B)-(D) over the phi nodes, k and n_phi - k together
    float R0c[LO + 1], R0s[LO + 1], P1c[LO + 1], P1s[LO + 1], P2c[LO + 1], P2s[LO + 1];
#pragma unroll
    for (int t = 0; t <= LO; ++t) R0c[t] = R0s[t] = P1c[t] = P1s[t] = P2c[t] = P2s[t] = 0.f;
    {
        float A = 0.f, B = 0.f, C = 0.f, a = 0.f, b = 0.f, c = 0.f;
#pragma unroll
        for (int t = 0; t <= L1; ++t) {
            A += Ac[t];
            if constexpr (SPIN) B += Bc[t], C += Cc[t];
        }
#pragma unroll
        for (int t = 0; t <= L2; ++t) {
            a += ac[t];
            if constexpr (SPIN) b += bc[t], c += cc[t];
        }
        float r0 = A * a, p1 = 0.f, p2 = 0.f;
        if constexpr (SPIN) {
            r0 = fmaf(B, b, fmaf(C, c, r0));
            p1 = fmaf(A, b, a * B);
            p2 = fmaf(A, c, a * C);
        }
#pragma unroll
        for (int t = 0; t <= LO; ++t) {
            R0c[t] += r0;
            if constexpr (SPIN) P1c[t] += p1, P2c[t] += p2;
        }
    }
#pragma unroll
    for (int k = 1; k <= S::KP; ++k) {
        const float* __restrict__ cs = g + Y.cosT + k * TM1;
        const float* __restrict__ sn = g + Y.sinT + k * TM1;
        float Ap, Am, ap, am;
        synth<L1>(Ac, As, cs, sn, Ap, Am);
        synth<L2>(ac, as, cs, sn, ap, am);
        float r0p = Ap * ap, r0m = Am * am, p1p = 0.f, p1m = 0.f, p2p = 0.f, p2m = 0.f;
        if constexpr (SPIN) {
            float Bp, Bm, Cp, Cm, bp, bm, cp, cm;
            synth<L1>(Bc, Bs, cs, sn, Bp, Bm);
            synth<L1>(Cc, Cs, cs, sn, Cp, Cm);
            synth<L2>(bc, bs, cs, sn, bp, bm);
            synth<L2>(cc, cs2, cs, sn, cp, cm);
            r0p = fmaf(Bp, bp, fmaf(Cp, cp, r0p));
            r0m = fmaf(Bm, bm, fmaf(Cm, cm, r0m));
            p1p = fmaf(Ap, bp, ap * Bp);
            p1m = fmaf(Am, bm, am * Bm);
            p2p = fmaf(Ap, cp, ap * Cp);
            p2m = fmaf(Am, cm, am * Cm);
        }
        const float sr = r0p + r0m, dr = r0p - r0m;
        R0c[0] += sr;
#pragma unroll
        for (int t = 1; t <= LO; ++t) {
            R0c[t] = fmaf(sr, cs[t], R0c[t]);
            R0s[t] = fmaf(dr, sn[t], R0s[t]);
        }
        if constexpr (SPIN) {
            const float s1 = p1p + p1m, q1 = p1p - p1m, s2 = p2p + p2m, q2 = p2p - p2m;
            P1c[0] += s1;
            P2c[0] += s2;
#pragma unroll
            for (int t = 1; t <= LO; ++t) {
                P1c[t] = fmaf(s1, cs[t], P1c[t]);
                P1s[t] = fmaf(q1, sn[t], P1s[t]);
                P2c[t] = fmaf(s2, cs[t], P2c[t]);
                P2s[t] = fmaf(q2, sn[t], P2s[t]);
            }
        }
    }
    if constexpr (S::NP % 2 == 0) {  // phi = pi: cos(t pi) = (-1)^t, sin = 0
        float A = 0.f, B = 0.f, C = 0.f, a = 0.f, b = 0.f, c = 0.f;
#pragma unroll
        for (int t = 0; t <= L1; ++t) {
            const float sg = (t & 1) ? -1.f : 1.f;
            A = fmaf(sg, Ac[t], A);
            if constexpr (SPIN) B = fmaf(sg, Bc[t], B), C = fmaf(sg, Cc[t], C);
        }
#pragma unroll
        for (int t = 0; t <= L2; ++t) {
            const float sg = (t & 1) ? -1.f : 1.f;
            a = fmaf(sg, ac[t], a);
            if constexpr (SPIN) b = fmaf(sg, bc[t], b), c = fmaf(sg, cc[t], c);
        }
        float r0 = A * a, p1 = 0.f, p2 = 0.f;
        if constexpr (SPIN) {
            r0 = fmaf(B, b, fmaf(C, c, r0));
            p1 = fmaf(A, b, a * B);
            p2 = fmaf(A, c, a * C);
        }
#pragma unroll
        for (int t = 0; t <= LO; ++t) {
            const float sg = (t & 1) ? -1.f : 1.f;
            R0c[t] = fmaf(sg, r0, R0c[t]);
            if constexpr (SPIN) P1c[t] = fmaf(sg, p1, P1c[t]), P2c[t] = fmaf(sg, p2, P2c[t]);
        }
    }

    // (E) publish this node's spectra, then every owner wave projects its groups
    //     onto the output coefficients, summing over the nodes in a fixed order.
    using SP = Spectra<LO, SPIN>;
    constexpr int BO = (LO + 1) * (LO + 1);
    float* D = X1 + (node * 64 + lane) * SP::DS;  // aliases the input tiles
    __syncthreads();                               // every wave is past step (A)
    if constexpr (SPIN) {
        R0c[0] = fmaf(-0.5f * S::NP, fmaf(d1, d2, e1 * e2), R0c[0]);
        // m3 = 0, |s3| = 1: sums over phi of Re/Im h+ and h-
        const float sP1 = 1.41421356237309505f * P1c[0];
        const float sP2 = 1.41421356237309505f * P2c[0];
        const float sP4 = -static_cast<float>(S::NP) * fmaf(d2, Ac[0], d1 * ac[0]);
        const float sP3 = static_cast<float>(S::NP) * fmaf(e2, Ac[0], e1 * ac[0]);
        const float v0 = 0.5f * (sP1 + sP4), v1 = 0.5f * (sP3 + sP2);
        const float v2 = 0.5f * (sP1 - sP4), v3 = 0.5f * (sP3 - sP2);
        const float* m0 = g + Y.m0;
        D[0] = R0c[0];
        D[1] = fmaf(m0[0], v0, fmaf(m0[1], v1, fmaf(m0[2], v2, m0[3] * v3)));
        D[2] = fmaf(m0[4], v0, fmaf(m0[5], v1, fmaf(m0[6], v2, m0[7] * v3)));
#pragma unroll
        for (int t = 1; t <= LO; ++t) {
            float* d = D + 3 + 6 * (t - 1);
            d[0] = R0c[t];
            d[1] = R0s[t];
            d[2] = P1c[t] + P2s[t];
            d[3] = P1c[t] - P2s[t];
            d[4] = P2c[t] - P1s[t];
            d[5] = -P2c[t] - P1s[t];
        }
    } else {
        D[0] = R0c[0];
#pragma unroll
        for (int t = 1; t <= LO; ++t) {
            D[1 + 2 * (t - 1)] = R0c[t];
            D[2 + 2 * (t - 1)] = R0s[t];
        }
    }
    __syncthreads();

    constexpr Owners<SP::NG> own = assign_owners<LO, SPIN, S::WAVES>();
    float* yr = YT + lane * S::STO;
#pragma unroll
    for (int gi = 0; gi < SP::NG; ++gi) {
        if (own.owner[gi] != node) continue;
        const int t = SP::t_of(gi), slot = SP::slot_of(gi);
        float dv[S::NT];
#pragma unroll
        for (int j = 0; j < S::NT; ++j) dv[j] = X1[(j * 64 + lane) * SP::DS + gi];
        // output block and table of this group
        int blk = 0, sgn = 1, tab_base = 0;
        bool e1z = false;
        if (t == 0) {
            if (slot == 0) { blk = SPIN ? 1 : 0; tab_base = Y.e0c; }
            else { blk = slot == 1 ? 2 : 0; e1z = true; tab_base = Y.e1z; }
        } else if (slot == 0) { blk = SPIN ? 1 : 0; tab_base = Y.e0c; }
        else if (slot == 1) { blk = SPIN ? 1 : 0; tab_base = Y.e0s; sgn = -1; }
        else if (slot == 2) { blk = 2; tab_base = Y.e1p; }
        else if (slot == 3) { blk = 0; tab_base = Y.e1m; }
        else if (slot == 4) { blk = 2; tab_base = Y.e1p; sgn = -1; }
        else { blk = 0; tab_base = Y.e1m; sgn = -1; }
#pragma unroll
        for (int l = SP::lmin(gi); l <= LO; ++l) {
            const int toff = e1z ? tab_base + l : tab_base + tri(LO, t, l);
            float acc = 0.f;
#pragma unroll
            for (int j = 0; j < S::NT; ++j) acc = fmaf(tab[Y.glob + j * Y.pb + toff], dv[j], acc);
            yr[blk * BO + l * l + l + sgn * t] = acc;
        }
    }
    __syncthreads();
    if constexpr (SPIN) {
        if (parity) {
            parity_mix_rows<LO>(YT, S::STO, nvalid, true, tid, S::THREADS);
            __syncthreads();
        }
    }
    store_tile<S::NCO, S::STO>(out + u0 * S::NCO, nvalid, YT, tid, S::THREADS);
}


template <int L, bool SPIN, typename TIO, bool BWD>
__global__ __launch_bounds__((PairShape<L, SPIN>::THREADS)) void spingtp_fwd_pair_kernel(
    const TIO* __restrict__ x1, const TIO* __restrict__ x2, TIO* __restrict__ out, int64_t units, int64_t cpx2,
    const float* __restrict__ tab) {
    using P = PairShape<L, SPIN>;
    constexpr Layout Y = P::Y;
    constexpr int TM1 = Y.TM + 1;
    constexpr int BO = (L + 1) * (L + 1);
    __shared__ float lds[P::LDS_FLOATS];
    float* X1 = lds;
    float* X2 = X1 + P::UNITS * P::ST;
    float* YT = lds + P::REGION;
    float* TR = YT + P::UNITS * P::ST;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int u = lane >> 1;
    const int sub = lane & 1;
    const int node = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t u0 = static_cast<int64_t>(blockIdx.x) * P::UNITS;
    const int nvalid = static_cast<int>(units - u0 < P::UNITS ? units - u0 : P::UNITS);
    const float* __restrict__ g = tab;

    for (int i = tid; i < P::UNITS * P::ST; i += P::THREADS) YT[i] = 0.f;
    for (int i = tid; i < P::TRIG; i += P::THREADS) {
        const int sb = i / (P::NP * (L + 1));
        const int r = i - sb * (P::NP * (L + 1));
        const int k = r / (L + 1), t = r - k * (L + 1);
        TR[i] = g[(sb ? Y.sinT : Y.cosT) + k * TM1 + t];
    }
    load_tile<P::NC, P::ST>(x1 + u0 * P::NC, nvalid, X1, tid, P::THREADS);
    if (cpx2 == 1)
        load_tile<P::NC, P::ST>(x2 + u0 * P::NC, nvalid, X2, tid, P::THREADS);
    else
        load_tile_shared<P::NC, P::ST>(x2, u0, nvalid, cpx2, X2, tid, P::THREADS);
    __syncthreads();
    bool parity = false;  // uniform
    if constexpr (SPIN) {
        parity = tab[Y.par] != 0.f;
        if (parity) {
            parity_mix_rows<L>(X1, P::ST, nvalid, false, tid, P::THREADS);
            parity_mix_rows<L>(X2, P::ST, nvalid, false, tid, P::THREADS);
            __syncthreads();
        }
    }

    const float* __restrict__ tb = tab + Y.glob + node * Y.pb;
    float Q0[L + 1], Q1[L + 1], Q2[L + 1], zslot;
    pair_spectra<L, SPIN, BWD>((sub ? X2 : X1) + u * P::ST, tb, g, TR + sub * (P::NP * (L + 1)), sub, Q0, Q1, Q2, zslot);
    __syncthreads();  // every wave is past step (A): the input tiles are free
    pair_publish<L, SPIN>(X1 + (node * P::UNITS + u) * P::DS, sub, Q0, Q1, Q2, zslot);
    __syncthreads();

    constexpr Owners<P::NG> own = assign_pair_owners<L, SPIN, P::WAVES>();
    float* yr = YT + u * P::ST;
#pragma unroll
    for (int gi = 0; gi < P::NG; ++gi) {
        if (own.owner[gi] != node) continue;
        const int t = P::t_of(gi), kind = P::kind_of(gi);
        float dv[P::NT];
#pragma unroll
        for (int j = 0; j < P::NT; ++j) dv[j] = X1[(j * P::UNITS + u) * P::DS + P::slot(gi) + sub];
        int tab_base = Y.e0c, blk = SPIN ? BO : 0;
        if (kind == 1) tab_base = Y.e1p, blk = 2 * BO;
        if (kind == 2) tab_base = Y.e1m, blk = 0;
        if (kind == 3) tab_base = Y.e1z, blk = sub ? 0 : 2 * BO;
        const bool write = !(t == 0 && kind == 0 && sub);
#pragma unroll
        for (int l = P::lmin(gi); l <= L; ++l) {
            const int toff = kind == 3 ? tab_base + l : tab_base + tri(L, t, l);
            float acc = 0.f;
#pragma unroll
            for (int j = 0; j < P::NT; ++j) acc = fmaf(tab[Y.glob + j * Y.pb + toff], dv[j], acc);
            if (write) yr[blk + l * l + l + (sub ? -t : t)] = acc;
        }
    }
    __syncthreads();
    if constexpr (SPIN) {
        if (parity) {
            parity_mix_rows<L>(YT, P::ST, nvalid, true, tid, P::THREADS);
            __syncthreads();
        }
    }
    store_tile<P::NC, P::ST>(out + u0 * P::NC, nvalid, YT, tid, P::THREADS);
}

template <int L, bool SPIN, typename TIO, bool BWD>
hipError_t launch_pair(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float* tab,
                       const uint32_t*, hipStream_t stream) {
    using P = PairShape<L, SPIN>;
    const int64_t blocks = (units + P::UNITS - 1) / P::UNITS;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((spingtp_fwd_pair_kernel<L, SPIN, TIO, BWD>), dim3(static_cast<unsigned>(blocks)),
                       dim3(P::THREADS), 0, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                       static_cast<TIO*>(out), units, cpx2, tab);
    return hipGetLastError();
}


template <int L1, int L2, int LO, bool SPIN, typename TIO>
hipError_t launch(const void* x1, const void* x2, void* out, int64_t units, int64_t cpx2, const float* tab,
                  const uint32_t*, hipStream_t stream) {
    using S = Shape<L1, L2, LO, SPIN>;
    const int64_t blocks = (units + 63) / 64;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((spingtp_fwd_kernel<L1, L2, LO, SPIN, TIO>), dim3(static_cast<unsigned>(blocks)),
                       dim3(S::THREADS), 0, stream, static_cast<const TIO*>(x1), static_cast<const TIO*>(x2),
                       static_cast<TIO*>(out), units, cpx2, tab);
    return hipGetLastError();
}

struct Registered {
    int L1, L2, LO, spin, dtype;
    KernelEntry entry;
    // bases served: -1 every basis (the tiles are mixed in LDS under the plan's
    // table flag, or there is no |s| = 1 sector), 0 the two paper bases, 1 the parity one
    int basis_par = -1;
};

template <int L1, int L2, int LO, bool SPIN, typename TIO>
constexpr Registered reg() {
    using S = Shape<L1, L2, LO, SPIN>;
    return Registered{L1, L2, LO, SPIN ? 1 : 0, sizeof(TIO) == 4 ? 0 : 1,
                      KernelEntry{S::WAVES, 64, static_cast<int>(S::LDS_FLOATS * sizeof(float)), 1,
                                  &launch<L1, L2, LO, SPIN, TIO>, &launch<L1, L2, LO, SPIN, TIO>}};
}

#define SPINGTP_REG(L1, L2, LO, SPIN) reg<L1, L2, LO, SPIN, float>(), reg<L1, L2, LO, SPIN, uint16_t>()

template <int L, bool SPIN, typename TIO>
constexpr Registered reg_pair() {
    using P = PairShape<L, SPIN>;
    return Registered{L, L, L, SPIN ? 1 : 0, sizeof(TIO) == 4 ? 0 : 1,
                      KernelEntry{P::WAVES, P::UNITS, static_cast<int>(P::LDS_FLOATS * sizeof(float)), 2,
                                  &launch_pair<L, SPIN, TIO, false>, &launch_pair<L, SPIN, TIO, true>}};
}
#define SPINGTP_REG_PAIR(L, SPIN) reg_pair<L, SPIN, float>(), reg_pair<L, SPIN, uint16_t>()

template <int L, bool SPIN, int W, typename TIO, bool PAR = false>
constexpr Registered reg_big() {
    using B = BigShape<L, SPIN, W>;
    return Registered{L, L, L, SPIN ? 1 : 0, sizeof(TIO) == 4 ? 0 : 1,
                      KernelEntry{B::WAVES, B::UNITS, static_cast<int>(B::LDS_FLOATS * sizeof(float)), 3,
                                  &launch_big<L, SPIN, W, false, PAR, TIO>, &launch_big<L, SPIN, W, true, PAR, TIO>},
                      SPIN ? (PAR ? 1 : 0) : -1};
}
// (the parity-basis instantiations with spins are in forward_big_parity.hip)
#define SPINGTP_REG_BIG(L)                                                                                        \
    reg_big<L, true, big_waves<L, true>(), float>(), reg_big<L, false, big_waves<L, false>(), float>(),          \
        reg_big<L, true, big_waves<L, true>(), uint16_t>(), reg_big<L, false, big_waves<L, false>(), uint16_t>()

const Registered kRegistry[] = {
    SPINGTP_REG(0, 0, 0, false), SPINGTP_REG(1, 1, 1, false), SPINGTP_REG(2, 2, 2, false),
    SPINGTP_REG(3, 3, 3, false), SPINGTP_REG(4, 4, 4, false), SPINGTP_REG(6, 6, 6, false),
    SPINGTP_REG(1, 1, 1, true),  SPINGTP_REG(2, 2, 2, true),  SPINGTP_REG(3, 3, 3, true),
    SPINGTP_REG(4, 4, 4, true),  SPINGTP_REG(5, 5, 5, true),  SPINGTP_REG(6, 6, 6, true),
    SPINGTP_REG(1, 3, 3, true),  SPINGTP_REG(2, 1, 3, true),  SPINGTP_REG(8, 8, 8, false),
    SPINGTP_REG_PAIR(7, true),   SPINGTP_REG_PAIR(8, true),   SPINGTP_REG_BIG(9),
    SPINGTP_REG_BIG(10),         SPINGTP_REG_BIG(11),         SPINGTP_REG_BIG(12),
    SPINGTP_REG_BIG(13),         SPINGTP_REG_BIG(14),         SPINGTP_REG_BIG(15),
    SPINGTP_REG_BIG(16),
};

}  // namespace

const KernelEntry* find_kernel(int L1, int L2, int LO, int spin_mode, int dtype, bool parity) {
    for (const Registered& r : kRegistry)
        if (r.L1 == L1 && r.L2 == L2 && r.LO == LO && r.spin == spin_mode && r.dtype == dtype &&
            (r.basis_par < 0 || r.basis_par == (parity ? 1 : 0)))
            return &r.entry;
    if (parity && spin_mode == 1 && L1 == L2 && L2 == LO) return find_big_parity_kernel(L1, dtype);
    return nullptr;
}

}  // namespace spingtp
