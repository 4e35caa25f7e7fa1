// Plan-table layout shared by the host plan builder and the device kernels.
//
// The quadrature grid is the exact tensor-product rule for the triple products
// s1Y s2Y conj(s3Y) with s3 = s1 + s2 (paper Sec. 3.2 eq. generalized_gaunt):
// the theta part is a polynomial in cos(theta) of degree <= L1+L2+Lout and the
// phi part a Fourier mode of order <= L1+L2+Lout, so
//   n_theta = ceil((L1+L2+Lout+1)/2) Gauss-Legendre nodes in cos(theta),
//   n_phi   = L1+L2+Lout+1 uniform nodes phi_k = 2 pi k / n_phi
// integrate the product exactly.
//
// Table block (fp32 on the device, float64 from spingtp_plan_tables_host):
//   global part (offsets from 0):
//     N0[4][2]   t = 0 mixing of the |s| = 1 sector on input:
//                (W+, W-) -> (B~c0, C~c0, delta, eps)
//     N0B[4][2]  the same for input 2 (absorbs conjugation on backward tables)
//     M0[2][4]   t = 0 mixing of the |s| = 1 sector on output:
//                (sum hR+, sum hI+, sum hR-, sum hI-) -> (Z+, Z-)
//     PAR[4]     PAR[0] = 1: the plan's basis is the parity-labelled one and the
//                kernels mix tiles by P on load and by P^T before the store
//     COS[n_phi][TM+1], SIN[n_phi][TM+1]   cos(t phi_k), sin(t phi_k)
//   then one block per theta node j (offset glob + j * pb):
//     A0C, A0S, AUP, AUM   triangles over (t, l), l >= t, degree LA = max(L1, L2)
//     AW[LA+1]
//     E0C, E0S, E1P, E1M   triangles over (t, l), degree Lout
//     E1Z[Lout+1]
//   with tri(L, t, l) = t (L+1) - t (t-1)/2 + (l - t).
#pragma once

namespace spingtp {

struct Layout {
    int L1, L2, LO, LA, TM, NT, NP;
    int triA, triO;
    int n0, n0b, m0, par, cosT, sinT, glob;
    int a0c, a0s, aup, aum, aw, e0c, e0s, e1p, e1m, e1z, pb;
    int total;
};

constexpr int round4(int v) { return (v + 3) & ~3; }
constexpr int imax(int a, int b) { return a > b ? a : b; }
constexpr int tri_size(int L) { return (L + 1) * (L + 2) / 2; }
__host__ __device__ constexpr int tri(int L, int t, int l) { return t * (L + 1) - t * (t - 1) / 2 + (l - t); }

__host__ __device__ constexpr Layout make_layout(int L1, int L2, int LO) {
    Layout y{};
    y.L1 = L1;
    y.L2 = L2;
    y.LO = LO;
    y.LA = imax(L1, L2);
    y.TM = imax(y.LA, LO);
    y.NT = (L1 + L2 + LO + 2) / 2;
    y.NP = L1 + L2 + LO + 1;
    y.triA = tri_size(y.LA);
    y.triO = tri_size(LO);
    y.n0 = 0;
    y.n0b = 8;
    y.m0 = 16;
    y.par = 24;  // 1: the plan's basis is the parity-labelled one (tiles are mixed on load and store)
    y.cosT = 28;
    y.sinT = y.cosT + y.NP * (y.TM + 1);
    y.glob = round4(y.sinT + y.NP * (y.TM + 1));
    y.a0c = 0;
    y.a0s = y.a0c + y.triA;
    y.aup = y.a0s + y.triA;
    y.aum = y.aup + y.triA;
    y.aw = y.aum + y.triA;
    y.e0c = y.aw + y.LA + 1;
    y.e0s = y.e0c + y.triO;
    y.e1p = y.e0s + y.triO;
    y.e1m = y.e1p + y.triO;
    y.e1z = y.e1m + y.triO;
    y.pb = round4(y.e1z + LO + 1);
    y.total = y.glob + y.NT * y.pb;
    return y;
}

}  // namespace spingtp
