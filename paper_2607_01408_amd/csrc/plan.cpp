// Host side of the SpinGTP library: argument checks, float64 plan tables, plan
// lifetime and the C ABI entry points other than the forward launch.
//
// The tables hold everything the forward kernel needs to evaluate the two input
// fields on the exact quadrature grid (layout.h), multiply them spin pair by spin
// pair, and project the products back (paper App. B proof: a path is two inverse
// transforms, a pointwise product and one forward transform).  The spin-weighted
// harmonics come from the explicit Goldberg sum (paper App. A.1), the real-basis
// maps from eq. real_swsh and App. C.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <map>
#include <set>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <utility>
#include <vector>

#include "internal.h"

namespace spingtp {
namespace {

constexpr double kPi = 3.14159265358979323846264338327950288;
constexpr double kSqrt2 = 1.41421356237309504880168872420969808;

double factorial(int n) {
    double f = 1.0;
    for (int i = 2; i <= n; ++i) f *= i;
    return f;
}

double binom(int n, int k) {
    if (k < 0 || k > n) return 0.0;
    double b = 1.0;
    for (int i = 1; i <= k; ++i) b = b * (n - k + i) / i;
    return std::round(b);
}

// sY_lm(theta, 0) from the Goldberg sum (App. A.1) in half-angle form,
// sin^{2l}(theta/2) cot^k(theta/2) = sin^{2l-k} cos^k, k = 2r + s - m, with the
// prefactor (-1)^{m+l-s} sqrt((l+m)!(l-m)!(2l+1) / (4 pi (l+s)!(l-s)!)) that
// reproduces the closed forms of 1Y10 and 1Y1(+-1) printed there.
double swsh_theta(int s, int l, int m, double theta) {
    if (std::abs(s) > l || std::abs(m) > l) return 0.0;
    const double c = std::cos(0.5 * theta), sn = std::sin(0.5 * theta);
    double sum = 0.0;
    for (int r = 0; r <= l - s; ++r) {
        const int j = r + s - m;
        if (j < 0 || j > l + s) continue;
        const int k = 2 * r + s - m;
        const double coef = ((r & 1) ? -1.0 : 1.0) * binom(l - s, r) * binom(l + s, j);
        sum += coef * std::pow(sn, 2 * l - k) * std::pow(c, k);
    }
    const double mag = std::sqrt((2 * l + 1) / (4.0 * kPi) * (factorial(l + m) * factorial(l - m)) /
                                 (factorial(l + s) * factorial(l - s)));
    const double sign = (((m + l - s) % 2) != 0) ? -1.0 : 1.0;
    return sign * mag * sum;
}

// Gauss-Legendre rule on [-1, 1] by Newton iteration on P_n (three-term
// recurrence), the classical method of e.g. Numerical Recipes "gauleg".
void gauss_legendre(int n, std::vector<double>& x, std::vector<double>& w) {
    x.assign(n, 0.0);
    w.assign(n, 0.0);
    for (int i = 0; i < n; ++i) {
        double z = std::cos(kPi * (i + 0.75) / (n + 0.5));
        double dp = 1.0;
        for (int it = 0; it < 100; ++it) {
            double p0 = 1.0, p1 = z;
            for (int k = 2; k <= n; ++k) {
                const double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
                p0 = p1;
                p1 = p2;
            }
            if (n == 1) p0 = 1.0, p1 = z;
            dp = n * (z * p1 - p0) / (z * z - 1.0);
            const double dz = p1 / dp;
            z -= dz;
            if (std::fabs(dz) < 1e-16) break;
        }
        double p0 = 1.0, p1 = z;
        for (int k = 2; k <= n; ++k) {
            const double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
            p0 = p1;
            p1 = p2;
        }
        dp = n * (z * p1 - p0) / (z * z - 1.0);
        x[i] = z;
        w[i] = 2.0 / ((1.0 - z * z) * dp * dp);
    }
}

// Complex entry Q[(s, 0), (sigma, 0)] of the real->complex map for |s| = 1 at
// m = 0 (App. C; eq. real_swsh sets sR_l0 = sY_l0, the paired reading mixes the
// two m = 0 slots).
struct Cplx {
    double re, im;
};
// s: the sign of the row's spin (+|sigma| or -|sigma|).
Cplx q_m0(unsigned flags, int s, int sigma) {
    const double h = 1.0 / kSqrt2;
    if (flags == SPINGTP_BASIS_REAL_PAPER) return ((s > 0) == (sigma > 0)) ? Cplx{1.0, 0.0} : Cplx{0.0, 0.0};
    // paired: column (+|s|,0) -> (h, (-1)^s h) on rows (+|s|,0), (-|s|,0);
    //         column (-|s|,0) -> (i h, -i (-1)^s h)
    const double sg = (std::abs(sigma) % 2) ? -1.0 : 1.0;
    if (sigma > 0) return (s > 0) ? Cplx{h, 0.0} : Cplx{sg * h, 0.0};
    return (s > 0) ? Cplx{0.0, h} : Cplx{0.0, -sg * h};
}

// Complex expansion of the real basis column (sigma, l, k) (eq. real_swsh, App. C):
// up to two entries (s, m, Q[(s,l,m),(sigma,l,k)]); returns their number.
struct QEnt {
    int s, m;
    Cplx q;
};
int real_column(int sigma, int k, unsigned flags, QEnt* e) {
    const double h = 1.0 / kSqrt2;
    if (k > 0) {
        e[0] = {sigma, k, {h, 0.0}};
        e[1] = {-sigma, -k, {(((k + sigma) % 2) != 0 ? -h : h), 0.0}};
        return 2;
    }
    if (k < 0) {
        const int a = -k;
        e[0] = {sigma, a, {0.0, h}};
        e[1] = {-sigma, k, {0.0, (((a + sigma) % 2) != 0 ? h : -h)}};
        return 2;
    }
    if (sigma == 0 || flags == SPINGTP_BASIS_REAL_PAPER) {
        e[0] = {sigma, 0, {1.0, 0.0}};
        return 1;
    }
    const int sa = std::abs(sigma);
    e[0] = {sa, 0, q_m0(flags, 1, sigma)};
    e[1] = {-sa, 0, q_m0(flags, -1, sigma)};
    return 2;
}

// The parity-labelled basis (Sec. 3.4 eq. parity_basis) is the paper's real
// basis followed by the orthogonal map P, x_real = P x_parity: per slot (l, m)
// with l >= |s| > 0, x[-s] = (c_+ + c_-)/sqrt2 and x[s] = (-1)^l (c_+ - c_-)/sqrt2,
// c_+ stored in the -|s| block and c_- in the +|s| block.  Every table of a
// parity plan is derived from the paper basis through P.
unsigned literal_basis(unsigned flags) {
    return flags == SPINGTP_BASIS_PARITY ? SPINGTP_BASIS_REAL_PAPER : flags;
}

// v <- P^T v (transpose = true) or v <- P v, along one axis of a strided array:
// element i of the axis sits at base + i * stride.
void parity_axis(double* base, size_t stride, int L, const int* spins, int n_spins, bool transpose) {
    const int nb = (L + 1) * (L + 1);
    const double h = 1.0 / kSqrt2;
    for (int a = 0; a < n_spins; ++a) {
        const int s = spins[a];
        if (s <= 0) continue;
        int b = -1;  // block of -s
        for (int i = 0; i < n_spins; ++i)
            if (spins[i] == -s) b = i;
        for (int l = s; l <= L; ++l) {
            const double t = (l % 2) ? -1.0 : 1.0;
            for (int m = -l; m <= l; ++m) {
                double& xm = base[(static_cast<size_t>(b) * nb + l * l + l + m) * stride];  // -s block
                double& xp = base[(static_cast<size_t>(a) * nb + l * l + l + m) * stride];  // +s block
                const double u = xm, v = xp;
                if (transpose) {
                    xm = (u + t * v) * h;
                    xp = (u - t * v) * h;
                } else {
                    xm = (u + v) * h;
                    xp = t * (u - v) * h;
                }
            }
        }
    }
}

}  // namespace

bool build_conj_map(int L, const int* spins, int n_spins, unsigned flags, std::vector<uint32_t>& out) {
    const int nb = (L + 1) * (L + 1);
    if (flags == SPINGTP_BASIS_PARITY) {
        // J_parity = P^T J P, again a signed permutation (or zero) row by row
        std::vector<uint32_t> lit;
        if (!build_conj_map(L, spins, n_spins, SPINGTP_BASIS_REAL_PAPER, lit)) return false;
        const size_t n = lit.size();
        std::vector<double> Jd(n * n, 0.0);
        for (size_t j = 0; j < n; ++j)
            if (!(lit[j] & kConjZero)) Jd[j * n + (lit[j] & 0xffffu)] = (lit[j] & kConjNeg) ? -1.0 : 1.0;
        // (J P)[r, :] = P^T applied to row r; then P^T (J P) column by column
        for (size_t r = 0; r < n; ++r) parity_axis(Jd.data() + r * n, 1, L, spins, n_spins, true);
        for (size_t c = 0; c < n; ++c) parity_axis(Jd.data() + c, n, L, spins, n_spins, true);
        out.assign(n, kConjZero);
        for (size_t j = 0; j < n; ++j) {
            int hits = 0;
            for (size_t i = 0; i < n; ++i) {
                const double v = Jd[j * n + i];
                if (std::fabs(v) < 1e-9) continue;
                if (std::fabs(std::fabs(v) - 1.0) > 1e-9) return false;
                out[j] = static_cast<uint32_t>(i) | (v < 0 ? kConjNeg : 0u);
                ++hits;
            }
            if (hits > 1) return false;
        }
        return true;
    }
    out.assign(static_cast<size_t>(n_spins) * nb, kConjZero);
    auto slot = [&](int si, int l, int k) { return si * nb + l * l + l + k; };
    for (int si = 0; si < n_spins; ++si)
        for (int l = std::abs(spins[si]); l <= L; ++l)
            for (int k = -l; k <= l; ++k) {
                // conjugated column: conj(sY_lm) = (-1)^(s+m) (-s)Y_l(-m) (App. A.1)
                QEnt e[2], c[2];
                const int n = real_column(spins[si], k, flags, e);
                for (int i = 0; i < n; ++i) {
                    const double sg = ((e[i].s + e[i].m) % 2 != 0) ? -1.0 : 1.0;
                    c[i] = {-e[i].s, -e[i].m, {sg * e[i].q.re, -sg * e[i].q.im}};
                }
                // the real column j with Q[:, j] = +-(conjugated column): J[j][k] = +-1
                bool found = false;
                for (int sj = 0; sj < n_spins && !found; ++sj) {
                    if (std::abs(spins[sj]) > l) continue;
                    for (int kj = -l; kj <= l && !found; ++kj) {
                        QEnt f[2];
                        const int nf = real_column(spins[sj], kj, flags, f);
                        if (nf != n) continue;
                        for (double sign : {1.0, -1.0}) {
                            bool all = true;
                            for (int i = 0; i < n && all; ++i) {
                                bool hit = false;
                                for (int q = 0; q < nf; ++q)
                                    hit |= f[q].s == c[i].s && f[q].m == c[i].m &&
                                           std::fabs(sign * f[q].q.re - c[i].q.re) < 1e-12 &&
                                           std::fabs(sign * f[q].q.im - c[i].q.im) < 1e-12;
                                all = hit;
                            }
                            if (all) {
                                // (J x)[j] = sign x[k]
                                out[slot(sj, l, kj)] = static_cast<uint32_t>(slot(si, l, k)) | (sign < 0 ? kConjNeg : 0u);
                                found = true;
                                break;
                            }
                        }
                    }
                }
                if (!found) return false;
            }
    return true;
}

bool build_tables(int L1, int L2, int LO, int spin_mode, unsigned flags, std::vector<double>& out,
                  bool conj_input2) {
    if (spin_mode > 1) return false;  // the Fourier kernels cover spins {0} and {-1, 0, +1}
    const Layout Y = make_layout(L1, L2, LO);
    out.assign(Y.total, 0.0);
    // a parity plan runs the paper basis's tables on tiles mixed by P (inputs) and
    // P^T (output); the conjugation folded below is then the paper basis's J,
    // since P^T J P x = P^T J (P x)
    out[Y.par] = (flags == SPINGTP_BASIS_PARITY && spin_mode == 1) ? 1.0 : 0.0;
    flags = literal_basis(flags);
    const double sq2 = kSqrt2;

    if (spin_mode == 1) {
        // Input, t = 0, |s| = 1: with W_sigma = sum_l x[sigma,l,0] Theta_{1,l,0} and
        // Theta_{-1,l,0} = -Theta_{1,l,0}, the m = 0 part of field f_s is
        // s * sum_sigma Q[(s,0),(sigma,0)] W_sigma.  The kernel keeps
        // B~c0 = sqrt2 (Re f+ + Re f-)/2, C~c0 = sqrt2 (Im f+ - Im f-)/2,
        // delta = Re f- - Re f+, eps = Im f- + Im f+.
        for (int col = 0; col < 2; ++col) {
            const int sigma = col == 0 ? 1 : -1;
            const Cplx qp = q_m0(flags, 1, sigma), qm = q_m0(flags, -1, sigma);
            const double Rp = qp.re, Ip = qp.im, Rm = -qm.re, Im_ = -qm.im;
            out[Y.n0 + 0 * 2 + col] = sq2 * (Rp + Rm) / 2.0;
            out[Y.n0 + 1 * 2 + col] = sq2 * (Ip - Im_) / 2.0;
            out[Y.n0 + 2 * 2 + col] = Rm - Rp;
            out[Y.n0 + 3 * 2 + col] = Im_ + Ip;
        }
        // Output, t = 0, |s| = 1: y[sigma,l,0] = Theta_{1,l,0} Re[conj(q(+,sigma)) h^+(0)
        // - conj(q(-,sigma)) h^-(0)], written on the sums of Re/Im h+- over phi.
        for (int row = 0; row < 2; ++row) {
            const int sigma = row == 0 ? 1 : -1;
            const Cplx qp = q_m0(flags, 1, sigma), qm = q_m0(flags, -1, sigma);
            out[Y.m0 + row * 4 + 0] = qp.re;
            out[Y.m0 + row * 4 + 1] = qp.im;
            out[Y.m0 + row * 4 + 2] = -qm.re;
            out[Y.m0 + row * 4 + 3] = -qm.im;
        }
    }
    // Input 2's copy of the N0 mixing.  For spingtp_backward input 2 enters
    // conjugated (J x2): J must act on the m = 0 slots of the |s| = 1 sectors only,
    // as (J x)[(sigma,l,0)] = sign_sigma x[(pi(sigma),l,0)] for every l, so that
    // W'_sigma = sign_sigma W_pi(sigma) folds into the two columns of N0.
    for (int i = 0; i < 8; ++i) out[Y.n0b + i] = out[Y.n0 + i];
    if (conj_input2) {
        const int s3[3] = {-1, 0, 1}, s1[1] = {0};
        std::vector<uint32_t> J;
        if (!build_conj_map(L2, spin_mode ? s3 : s1, spin_mode ? 3 : 1, flags, J)) return false;
        const int nb = (L2 + 1) * (L2 + 1);
        int pi[2] = {0, 1};
        double sg[2] = {1.0, 1.0};
        for (int j = 0; j < static_cast<int>(J.size()); ++j) {
            if (J[j] & kConjZero) continue;
            const int si = j / nb, r = j % nb, l = static_cast<int>(std::sqrt(static_cast<double>(r)) + 1e-9);
            const bool m0_spin = spin_mode == 1 && si != 1 && r == l * l + l;
            const int src = static_cast<int>(J[j] & 0xffffu);
            const double sign = (J[j] & kConjNeg) ? -1.0 : 1.0;
            if (!m0_spin) {
                if (src != j || sign != 1.0) return false;
                continue;
            }
            // column 0 of N0 is sigma = +1 (spin block 2), column 1 is sigma = -1 (block 0)
            const int col = si == 2 ? 0 : 1;
            const int ssi = src / nb, sr = src % nb;
            if (sr != r || ssi == 1) return false;
            const int scol = ssi == 2 ? 0 : 1;
            if (l == 1) {
                pi[col] = scol;
                sg[col] = sign;
            } else if (pi[col] != scol || sg[col] != sign) {
                return false;
            }
        }
        double n0b[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int q = 0; q < 4; ++q)
            for (int c = 0; c < 2; ++c) n0b[2 * q + pi[c]] += out[Y.n0 + 2 * q + c] * sg[c];
        for (int i = 0; i < 8; ++i) out[Y.n0b + i] = n0b[i];
    }

    for (int k = 0; k < Y.NP; ++k) {
        for (int t = 0; t <= Y.TM; ++t) {
            const double ang = 2.0 * kPi * static_cast<double>((k * t) % Y.NP) / Y.NP;
            out[Y.cosT + k * (Y.TM + 1) + t] = std::cos(ang);
            out[Y.sinT + k * (Y.TM + 1) + t] = std::sin(ang);
        }
    }
    std::vector<double> gx, gw;
    gauss_legendre(Y.NT, gx, gw);
    const double cphi = 2.0 * kPi / Y.NP;
    double wsum = 0.0;
    for (int j = 0; j < Y.NT; ++j) {
        const double th = std::acos(gx[j]);
        const double wc = gw[j] * cphi;
        wsum += gw[j];
        double* b = out.data() + Y.glob + static_cast<size_t>(j) * Y.pb;
        for (int t = 0; t <= Y.LA; ++t) {
            for (int l = t; l <= Y.LA; ++l) {
                const double th0 = swsh_theta(0, l, t, th);
                b[Y.a0c + tri(Y.LA, t, l)] = (t == 0 ? 1.0 : sq2) * th0;
                if (t > 0) b[Y.a0s + tri(Y.LA, t, l)] = -sq2 * th0;
                if (spin_mode == 1 && t > 0) {
                    b[Y.aup + tri(Y.LA, t, l)] = swsh_theta(1, l, t, th);
                    b[Y.aum + tri(Y.LA, t, l)] = swsh_theta(-1, l, t, th);
                }
            }
        }
        if (spin_mode == 1)
            for (int l = 1; l <= Y.LA; ++l) b[Y.aw + l] = swsh_theta(1, l, 0, th);
        for (int t = 0; t <= LO; ++t) {
            for (int l = t; l <= LO; ++l) {
                const double th0 = swsh_theta(0, l, t, th);
                b[Y.e0c + tri(LO, t, l)] = wc * (t == 0 ? 1.0 : sq2) * th0;
                if (t > 0) b[Y.e0s + tri(LO, t, l)] = -wc * sq2 * th0;
                if (spin_mode == 1 && t > 0) {
                    b[Y.e1p + tri(LO, t, l)] = wc * swsh_theta(1, l, t, th);
                    b[Y.e1m + tri(LO, t, l)] = wc * swsh_theta(-1, l, t, th);
                }
            }
        }
        if (spin_mode == 1)
            for (int l = 1; l <= LO; ++l) b[Y.e1z + l] = wc * swsh_theta(1, l, 0, th);
    }

    // Self-checks: the weights integrate 1 exactly, and the rule reproduces the
    // orthonormality of the highest-degree harmonics whose squares (degree 2l in
    // cos theta) it integrates exactly: l <= NT - 1.  The triple products of the
    // operation have degree L1 + L2 + Lout <= 2 NT - 1, which may be below 2 Lmax
    // when one degree exceeds the sum of the other two.
    if (std::fabs(wsum - 2.0) > 1e-13) return false;
    const int lmax = std::min(Y.TM, Y.NT - 1);
    for (int s = 0; s <= spin_mode; ++s) {
        for (int m = 0; m <= lmax; m += (lmax > 0 ? lmax : 1)) {
            for (int l = std::max(std::abs(s), m); l <= lmax; ++l) {
                double g = 0.0;
                for (int j = 0; j < Y.NT; ++j) {
                    const double v = swsh_theta(s, l, m, std::acos(gx[j]));
                    g += gw[j] * 2.0 * kPi * v * v;
                }
                if (std::fabs(g - 1.0) > 1e-10) return false;
            }
        }
    }
    return true;
}

// Operand tables of the matrix-core kernel (forward_mfma.hip), as packed fp16
// words (element 2w in the low half of word w).  fp32 values are split as
// hi = fp16(v), lo = fp16(v - hi), both rounded to nearest.
//   TB, 64 lanes x 8 words: lane l is row l % 32 of the step-(B) table (the phi
//     point phi_k, k = row, zero for k >= n_phi) and its K elements
//     8 (l / 32) + e, e = 0..7, are kappa = 8 (l / 32) + e: cos(kappa phi_k) for
//     kappa <= min(L, 7), sin((kappa - 8) phi_k) for 1 <= kappa - 8 <= L, and for
//     L = 8 sin(8 phi_k) at kappa = 8 (the slot sin 0 leaves free), else 0.
//     Words 0..3 hold hi, 4..7 lo.
//   TD[type][block], 2 x NB blocks of 64 lanes x 8 words: lane l is row
//     r' = l % 32 = 8i + 4h' + r of the step-(D) table, the spectrum t' = 4i + r
//     (zero for t' > L); K element e of lane l in block b is the point held by
//     step-(B) accumulator position v = 8b + e of half h'' = l / 32, i.e.
//     k = 8 (v / 4) + 4 h'' + v % 4 (zero for k >= n_phi).  Type 0 (R0, P1) rows
//     with h' = 0 are cos(t' phi_k) and with h' = 1 sin(t' phi_k); type 1 (P2)
//     swaps the two; the t' = 0 rows are cos 0 = 1 in both halves.
//   TB2a, TB2b (L = 8 only), after the TD blocks: the second K block of step (B)
//     for input 1 and input 2.  Its operand carries cos 8 of each lane's own input
//     in K element 0, i.e. input 1's at kappa 16 (lanes 0..31) and input 2's at
//     kappa 24 (lanes 32..63); TB2a has cos(8 phi_k) at kappa 16 only, TB2b at
//     kappa 24 only, so one operand serves both inputs.
void build_mfma_operands(int L, std::vector<uint32_t>& out) {
    const int NP = 3 * L + 1;
    const int NB = (NP + 15) / 16;
    const int KB2 = L >= 8 ? 2 : 0;  // second-K-block tables of step (B)
    out.assign(static_cast<size_t>(1 + 2 * NB + KB2) * 512, 0u);
    auto trig = [&](bool cosine, int t, int k) {
        const double ang = 2.0 * kPi * static_cast<double>((k * t) % NP) / NP;
        return cosine ? std::cos(ang) : std::sin(ang);
    };
    auto put = [&](size_t word0, int e, double v) {
        const _Float16 hi = static_cast<_Float16>(v);
        const _Float16 lo = static_cast<_Float16>(v - static_cast<double>(hi));
        uint16_t bh, bl;
        std::memcpy(&bh, &hi, 2);
        std::memcpy(&bl, &lo, 2);
        const int sh = 16 * (e & 1);
        out[word0 + e / 2] |= static_cast<uint32_t>(bh) << sh;
        out[word0 + 4 + e / 2] |= static_cast<uint32_t>(bl) << sh;
    };
    for (int lane = 0; lane < 64; ++lane) {
        const int k = lane % 32, half = lane / 32;
        for (int e = 0; e < 8; ++e) {
            const int kappa = 8 * half + e;
            double v = 0.0;
            if (k < NP) {
                if (kappa < 8 && kappa <= L) v = trig(true, kappa, k);
                if (kappa >= 9 && kappa - 8 <= L) v = trig(false, kappa - 8, k);
                if (kappa == 8 && L >= 8) v = trig(false, 8, k);
            }
            put(static_cast<size_t>(lane) * 8, e, v);
        }
    }
    for (int b = 0; b < KB2; ++b)  // b = 0: input 1 (lanes 0..31), b = 1: input 2 (lanes 32..63)
        for (int row = 0; row < NP; ++row)
            put(static_cast<size_t>(1 + 2 * NB + b) * 512 + static_cast<size_t>(32 * b + row) * 8, 0,
                trig(true, 8, row));
    for (int type = 0; type < 2; ++type)
        for (int b = 0; b < NB; ++b)
            for (int lane = 0; lane < 64; ++lane) {
                const int rr = lane % 32;
                const int i = rr / 8, hp = (rr / 4) % 2, r = rr % 4;
                const int tp = 4 * i + r;
                const size_t w0 = 512 + (static_cast<size_t>(type * NB + b) * 64 + lane) * 8;
                for (int e = 0; e < 8; ++e) {
                    const int v = 8 * b + e;
                    const int k = 8 * (v / 4) + 4 * (lane / 32) + v % 4;
                    double val = 0.0;
                    if (tp <= L && k < NP) {
                        const bool cosine = tp == 0 || (type == 0 ? hp == 0 : hp == 1);
                        val = trig(cosine, tp, k);
                    }
                    put(w0, e, val);
                }
            }
}

namespace {

// One contraction row of the precontracted kernel: x1 slot k1, and (for the
// per-channel weighted table) the path's input-2 and output blocks that the row's
// entries are restricted to (-1: no restriction).
struct PreRow {
    int k1, b2, b3, path;
};

// The item table of the precontracted kernel for the given contraction rows (see
// build_pre_tables): entry (q, k3) = sum over k2 of T[k1(q), k2, k3] x2[k2].
bool pre_table_from_rows(const std::vector<double>& T, int nc1, int nc2, int nco, int blk1, int n_spins,
                         const std::vector<PreRow>& rows, int ks, const std::vector<int>& blk2,
                         const std::vector<int>& blko, const std::vector<uint32_t>* J, int npaths,
                         std::vector<uint32_t>& out) {
    const int nt = (nco + 15) / 16, kst = 16 * ks + 4;
    // k3 rows per block: the whole kernel, or blocks of kPreBlockRows for the
    // large instantiations (KS or NT above 5); the weighted kernel always takes one block
    const int rb = ((ks > 5 || nt > 5) && npaths == 0) ? kPreBlockRows : 16 * nt;
    const int nb3 = (16 * nt + rb - 1) / rb;
    if (static_cast<int64_t>(rb) * kst > 0xffff) return false;  // 16-bit entry positions
    struct Entry {
        int dst;
        std::vector<std::pair<int, float>> items;
    };
    std::vector<std::vector<Entry>> entries(nb3);
    for (int q = 0; q < static_cast<int>(rows.size()); ++q) {
        const PreRow& rw = rows[q];
        for (int k3 = 0; k3 < nco; ++k3) {
            if (rw.b3 >= 0 && blko[k3] != rw.b3) continue;
            const int b = k3 / rb;
            Entry e{(k3 - b * rb) * kst + q, {}};
            for (int k2 = 0; k2 < nc2; ++k2) {
                if (rw.b2 >= 0 && blk2[k2] != rw.b2) continue;
                const double v = T[(static_cast<size_t>(rw.k1) * nc2 + k2) * nco + k3];
                if (std::fabs(v) <= 1e-12) continue;
                if (J != nullptr) {
                    if ((*J)[k2] & kConjZero) continue;  // J x2 is 0 there
                    const double sign = ((*J)[k2] & kConjNeg) ? -1.0 : 1.0;
                    e.items.emplace_back(static_cast<int>((*J)[k2] & 0xffffu), static_cast<float>(sign * v));
                } else {
                    e.items.emplace_back(k2, static_cast<float>(v));
                }
            }
            if (!e.items.empty()) entries[b].push_back(std::move(e));
        }
    }
    // per block: longest-first greedy balance of whole entries over the threads
    std::vector<std::vector<std::vector<const Entry*>>> per(nb3, std::vector<std::vector<const Entry*>>(kPreThreads));
    // the blocked kernel loads 16 items ahead without conditions: IPT a multiple
    // of 16 and 16 zero items after each block; the other kernel: multiple of 8
    const bool blocked = nb3 > 1 || rb != 16 * nt;
    const size_t quantum = blocked ? 16 : 8;
    size_t ipt = quantum;
    for (int b = 0; b < nb3; ++b) {
        std::stable_sort(entries[b].begin(), entries[b].end(),
                         [](const Entry& a, const Entry& c) { return a.items.size() > c.items.size(); });
        std::vector<size_t> load(kPreThreads, 0);
        for (const Entry& e : entries[b]) {
            const size_t t = static_cast<size_t>(std::min_element(load.begin(), load.end()) - load.begin());
            per[b][t].push_back(&e);
            load[t] += e.items.size();
        }
        ipt = std::max(ipt, (*std::max_element(load.begin(), load.end()) + quantum - 1) / quantum * quantum);
    }
    const size_t stride = blocked ? ipt + 16 : ipt;  // items per thread and block
    const size_t item_words = 2 * nb3 * stride * kPreThreads;
    out.assign(kPreHeader + item_words + (npaths > 0 ? rows.size() : 0), 0u);  // padding items: value 0
    out[0] = static_cast<uint32_t>(rows.size());
    out[1] = static_cast<uint32_t>(nc2);
    out[2] = static_cast<uint32_t>(nco);
    out[3] = static_cast<uint32_t>(blk1);
    out[4] = static_cast<uint32_t>(ks);
    out[5] = static_cast<uint32_t>(nt);
    out[6] = static_cast<uint32_t>(ipt);
    out[7] = static_cast<uint32_t>(kst);
    out[8] = static_cast<uint32_t>(nb3);
    out[9] = static_cast<uint32_t>(rb);
    out[10] = static_cast<uint32_t>(stride);
    out[11] = static_cast<uint32_t>(n_spins);
    out[12] = static_cast<uint32_t>(nc1);
    out[13] = static_cast<uint32_t>(npaths);
    out[14] = npaths > 0 ? static_cast<uint32_t>(kPreHeader + item_words) : 0u;
    for (int b = 0; b < nb3; ++b) {
        uint32_t* items = out.data() + kPreHeader + 2 * static_cast<size_t>(b) * stride * kPreThreads;
        for (int t = 0; t < kPreThreads; ++t) {
            size_t i = 0;
            for (const Entry* e : per[b][t])
                for (size_t j = 0; j < e->items.size(); ++j, ++i) {
                    const bool last = j + 1 == e->items.size();
                    uint32_t* it = items + 2 * (i * kPreThreads + t);
                    it[0] = static_cast<uint32_t>(e->dst) | (static_cast<uint32_t>(e->items[j].first) << 16) |
                            (last ? 1u << 24 : 0u);
                    std::memcpy(&it[1], &e->items[j].second, 4);
                }
        }
    }
    if (npaths > 0)  // the contraction rows: x1 slot | path << 16
        for (size_t q = 0; q < rows.size(); ++q)
            out[kPreHeader + item_words + q] =
                static_cast<uint32_t>(rows[q].k1) | (static_cast<uint32_t>(rows[q].path) << 16);
    return true;
}

}  // namespace

bool build_pre_tables(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                      std::vector<uint32_t>& out, bool conj_x2, const std::vector<double>* dense) {
    std::vector<double> own;
    if (dense == nullptr) build_dense_tensor(L1, L2, LO, spins, n_spins, flags, own);
    const std::vector<double>& T = dense != nullptr ? *dense : own;
    // conj_x2: the kernel reads x2 but must use J x2 (spingtp_backward_v1), so
    // each item's k2 becomes J's source slot and its value takes J's sign
    std::vector<uint32_t> J;
    if (conj_x2 && !build_conj_map(L2, spins, n_spins, flags, J)) return false;
    const int nc1 = n_spins * (L1 + 1) * (L1 + 1), nc2 = n_spins * (L2 + 1) * (L2 + 1);
    const int nco = n_spins * (LO + 1) * (LO + 1);
    std::vector<PreRow> rows(nc1);
    for (int k1 = 0; k1 < nc1; ++k1) rows[k1] = {k1, -1, -1, 0};
    return pre_table_from_rows(T, nc1, nc2, nco, (L1 + 1) * (L1 + 1), n_spins, rows, (nc1 + 15) / 16, {}, {},
                               conj_x2 ? &J : nullptr, 0, out);
}

bool build_pre_tables_channel_weighted(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                                       int ks, std::vector<uint32_t>& out, int* n_rows) {
    std::vector<double> T;
    build_dense_tensor(L1, L2, LO, spins, n_spins, flags, T);
    std::vector<std::array<int, 3>> paths;
    tensor_paths(L1, L2, LO, spins, n_spins, T, paths);
    const std::vector<int> b1 = slot_blocks(L1, spins, n_spins), b2 = slot_blocks(L2, spins, n_spins),
                           bo = slot_blocks(LO, spins, n_spins);
    std::vector<PreRow> rows;
    for (int p = 0; p < static_cast<int>(paths.size()); ++p)
        for (int k1 = 0; k1 < static_cast<int>(b1.size()); ++k1)
            if (b1[k1] == paths[p][0]) rows.push_back({k1, paths[p][1], paths[p][2], p});
    *n_rows = static_cast<int>(rows.size());
    if (static_cast<int>(rows.size()) > 16 * ks || static_cast<int>(b1.size()) > 16 * ks || paths.size() > 0xffff)
        return false;
    const int nc1 = static_cast<int>(b1.size()), nc2 = static_cast<int>(b2.size()), nco = static_cast<int>(bo.size());
    return pre_table_from_rows(T, nc1, nc2, nco, (L1 + 1) * (L1 + 1), n_spins, rows, ks, b2, bo, nullptr,
                               static_cast<int>(paths.size()), out);
}

bool build_bwd_v1w_table(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                         std::vector<uint32_t>& out, Bw1wShape* shape, const std::vector<double>* dense) {
    std::vector<double> own;
    if (dense == nullptr) build_dense_tensor(L1, L2, LO, spins, n_spins, flags, own);
    const std::vector<double>& T = dense != nullptr ? *dense : own;
    std::vector<std::array<int, 3>> paths;
    tensor_paths(L1, L2, LO, spins, n_spins, T, paths);
    const std::vector<int> b1 = slot_blocks(L1, spins, n_spins), b2 = slot_blocks(L2, spins, n_spins),
                           b3 = slot_blocks(LO, spins, n_spins);
    const int nc1 = static_cast<int>(b1.size()), nc2 = static_cast<int>(b2.size()), nco = static_cast<int>(b3.size());
    const int np = static_cast<int>(paths.size());
    if (std::max(std::max(nc1, nc2), std::max(nco, np)) > kBw1wMaxIndex) return false;
    auto st = [](int n) { return (n + 1) | 1; };
    const int lds = 64 * (2 * st(np) + st(nc1) + st(nco)) + st(nc2);
    if (lds > kBw1wMaxLdsFloats) return false;
    struct Ent {
        int k1, k2, k3, p;
        float v;
    };
    std::vector<Ent> ents;
    std::map<std::array<int, 3>, int> index;
    for (int p = 0; p < np; ++p) index[paths[p]] = p;
    for (int k1 = 0; k1 < nc1; ++k1)
        for (int k2 = 0; k2 < nc2; ++k2)
            for (int k3 = 0; k3 < nco; ++k3) {
                const double v = T[(static_cast<size_t>(k1) * nc2 + k2) * nco + k3];
                if (std::fabs(v) <= 1e-12) continue;  // quadrature round-off of an exact zero
                ents.push_back({k1, k2, k3, index.at({b1[k1], b2[k2], b3[k3]}), static_cast<float>(v)});
            }
    // one list: entries grouped by key (stable, so ascending (k1, k2, k3) inside a
    // group), each group padded to a multiple of 8 with zero-column entries
    struct List {
        std::vector<uint32_t> seg, words;
    };
    auto make = [&](int nkeys, auto key, auto fields, std::array<int, 3> pad) {
        List l;
        std::vector<std::vector<const Ent*>> by(nkeys);
        for (const Ent& e : ents) by[key(e)].push_back(&e);
        auto put = [&](std::array<int, 3> f, float v) {
            l.words.push_back(static_cast<uint32_t>(f[0]) | (static_cast<uint32_t>(f[1]) << 10) |
                              (static_cast<uint32_t>(f[2]) << 20));
            uint32_t bits = 0;
            std::memcpy(&bits, &v, 4);
            l.words.push_back(bits);
        };
        uint32_t at = 0;
        for (int k = 0; k < nkeys; ++k) {
            l.seg.push_back(at);
            for (const Ent* e : by[k]) put(fields(*e), e->v);
            size_t n = by[k].size();
            for (; n % 8 != 0; ++n) put(pad, 0.f);
            at += static_cast<uint32_t>(n);
        }
        l.seg.push_back(at);
        for (int i = 0; i < 96; ++i) put(pad, 0.f);  // read by the kernel's last prefetches
        return l;
    };
    const List l1 = make(
        nc1, [](const Ent& e) { return e.k1; }, [](const Ent& e) { return std::array<int, 3>{e.p, e.k2, e.k3}; },
        {np, nc2, nco});
    const List l2 = make(
        nc2, [](const Ent& e) { return e.k2; }, [](const Ent& e) { return std::array<int, 3>{e.p, e.k1, e.k3}; },
        {np, nc1, nco});
    const List lp = make(
        np, [](const Ent& e) { return e.p; }, [](const Ent& e) { return std::array<int, 3>{e.k1, e.k2, e.k3}; },
        {nc1, nc2, nco});
    const List l3 = make(
        nco, [](const Ent& e) { return e.k3; }, [](const Ent& e) { return std::array<int, 3>{e.p, e.k1, e.k2}; },
        {np, nc1, nc2});
    out.assign(40, 0u);
    out[0] = static_cast<uint32_t>(nc1);
    out[1] = static_cast<uint32_t>(nc2);
    out[2] = static_cast<uint32_t>(nco);
    out[3] = static_cast<uint32_t>(np);
    out[4] = static_cast<uint32_t>(ents.size());
    const List* lists[4] = {&l1, &l2, &lp, &l3};
    for (int i = 0; i < 4; ++i) {  // the waves' key ranges: about equal entry counts
        const std::vector<uint32_t>& sg = lists[i]->seg;
        const int nkeys = static_cast<int>(sg.size()) - 1;
        uint32_t* kr = out.data() + 16 + 5 * i;
        kr[0] = 0;
        kr[kBw1wWaves] = static_cast<uint32_t>(nkeys);
        for (int w = 1; w < kBw1wWaves; ++w) {
            const uint64_t target = static_cast<uint64_t>(sg[nkeys]) * w / kBw1wWaves;
            int k = static_cast<int>(kr[w - 1]);
            while (k < nkeys && sg[k] < target) ++k;
            kr[w] = static_cast<uint32_t>(k);
        }
    }
    const int seg_at[4] = {5, 6, 7, 11}, list_at[4] = {8, 9, 10, 12};
    for (int i = 0; i < 4; ++i) {
        out[seg_at[i]] = static_cast<uint32_t>(out.size());
        out.insert(out.end(), lists[i]->seg.begin(), lists[i]->seg.end());
    }
    for (int i = 0; i < 4; ++i) {
        out.resize((out.size() + 1) & ~size_t{1});  // 8-byte aligned entries
        out[list_at[i]] = static_cast<uint32_t>(out.size());
        out.insert(out.end(), lists[i]->words.begin(), lists[i]->words.end());
    }
    // the per-unit forms (x2 per unit): the gradients add x2 and gx2 tiles, the
    // forward holds the weight, x1, x2 and output tiles; 0 where they do not fit
    const int lds_unit_bwd = 64 * (2 * st(np) + st(nc1) + st(nco) + 2 * st(nc2));
    const int lds_unit_fwd = 64 * (st(np) + st(nc1) + st(nc2) + st(nco));
    const int lds_shared_fwd = 64 * (st(np) + st(nc1) + st(nco)) + st(nc2);
    if (shape != nullptr)
        *shape = Bw1wShape{nc1, nc2, nco, np, lds, lds_unit_bwd <= kBw1wMaxLdsFloats ? lds_unit_bwd : 0,
                           lds_unit_fwd <= kBw1wMaxLdsFloats ? lds_unit_fwd : 0,
                           lds_shared_fwd <= kBw1wMaxLdsFloats ? lds_shared_fwd : 0};
    return true;
}

// Dense real tensor T[k1][k2][k3] = Re sum conj(Q3) G Q1 Q2 (see spingtp.h).
// G^{(l3,m3,s3)}_{(l1,m1,s1)(l2,m2,s2)} = 2 pi sum_j w_j Y1(theta_j) Y2(theta_j) Y3(theta_j) for
// s3 = s1 + s2, m3 = m1 + m2 (the phi integral of the other combinations vanishes), on the
// Gauss-Legendre rule of the plan, which is exact for these triple products.
void build_dense_tensor(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                        std::vector<double>& T) {
    const int nb1 = (L1 + 1) * (L1 + 1), nb2 = (L2 + 1) * (L2 + 1), nbo = (LO + 1) * (LO + 1);
    if (flags == SPINGTP_BASIS_PARITY) {
        // T_parity[k1,k2,k3] = sum P[a,k1] P[b,k2] P[c,k3] T[a,b,c]: P^T along each axis
        build_dense_tensor(L1, L2, LO, spins, n_spins, SPINGTP_BASIS_REAL_PAPER, T);
        const size_t n1 = static_cast<size_t>(n_spins) * nb1, n2 = static_cast<size_t>(n_spins) * nb2,
                     n3 = static_cast<size_t>(n_spins) * nbo;
        for (size_t i = 0; i < n1 * n2; ++i) parity_axis(T.data() + i * n3, 1, LO, spins, n_spins, true);
        for (size_t i = 0; i < n1; ++i)
            for (size_t c = 0; c < n3; ++c)
                parity_axis(T.data() + i * n2 * n3 + c, n3, L2, spins, n_spins, true);
        for (size_t r = 0; r < n2 * n3; ++r) parity_axis(T.data() + r, n2 * n3, L1, spins, n_spins, true);
        return;
    }
    const size_t nc1 = static_cast<size_t>(n_spins) * nb1, nc2 = static_cast<size_t>(n_spins) * nb2,
                 nco = static_cast<size_t>(n_spins) * nbo;
    T.assign(nc1 * nc2 * nco, 0.0);
    const Layout Y = make_layout(L1, L2, LO);
    std::vector<double> gx, gw;
    gauss_legendre(Y.NT, gx, gw);
    const int LM = std::max(std::max(L1, L2), LO);
    auto sidx = [&](int s) {
        for (int i = 0; i < n_spins; ++i)
            if (spins[i] == s) return i;
        return -1;
    };
    // Theta tables [spin index][l][m + LM][node]
    std::vector<double> th(static_cast<size_t>(n_spins) * (LM + 1) * (2 * LM + 1) * Y.NT, 0.0);
    auto TH = [&](int si, int l, int m, int j) -> double& {
        return th[((static_cast<size_t>(si) * (LM + 1) + l) * (2 * LM + 1) + (m + LM)) * Y.NT + j];
    };
    for (int si = 0; si < n_spins; ++si)
        for (int l = std::abs(spins[si]); l <= LM; ++l)
            for (int m = -l; m <= l; ++m)
                for (int j = 0; j < Y.NT; ++j) TH(si, l, m, j) = swsh_theta(spins[si], l, m, std::acos(gx[j]));
    using Ent = QEnt;
    auto column = [&](int sigma, int k, Ent* e) -> int { return real_column(sigma, k, flags, e); };
    auto cmul = [](Cplx a, Cplx b) { return Cplx{a.re * b.re - a.im * b.im, a.re * b.im + a.im * b.re}; };
    // loop over real (k1, k2) and complex expansions; G picks m3 = m1 + m2, s3 = s1 + s2
    for (int i1 = 0; i1 < n_spins; ++i1)
        for (int l1 = std::abs(spins[i1]); l1 <= L1; ++l1)
            for (int k1 = -l1; k1 <= l1; ++k1) {
                Ent e1[2];
                const int n1 = column(spins[i1], k1, e1);
                const size_t c1 = static_cast<size_t>(i1) * nb1 + l1 * l1 + l1 + k1;
                for (int i2 = 0; i2 < n_spins; ++i2)
                    for (int l2 = std::abs(spins[i2]); l2 <= L2; ++l2)
                        for (int k2 = -l2; k2 <= l2; ++k2) {
                            Ent e2[2];
                            const int n2 = column(spins[i2], k2, e2);
                            const size_t c2 = static_cast<size_t>(i2) * nb2 + l2 * l2 + l2 + k2;
                            double* trow = T.data() + (c1 * nc2 + c2) * nco;
                            for (int a = 0; a < n1; ++a)
                                for (int b = 0; b < n2; ++b) {
                                    const int s3 = e1[a].s + e2[b].s, m3 = e1[a].m + e2[b].m;
                                    const int i3 = sidx(s3);
                                    if (i3 < 0) continue;
                                    const int ia = sidx(e1[a].s), ib = sidx(e2[b].s);
                                    const Cplx qq = cmul(e1[a].q, e2[b].q);
                                    const int l3lo = std::max(std::max(std::abs(s3), std::abs(m3)), std::abs(l1 - l2));
                                    for (int l3 = l3lo; l3 <= std::min(LO, l1 + l2); ++l3) {
                                        double gint = 0.0;
                                        for (int j = 0; j < Y.NT; ++j)
                                            gint += gw[j] * TH(ia, l1, e1[a].m, j) * TH(ib, l2, e2[b].m, j) *
                                                    TH(i3, l3, m3, j);
                                        gint *= 2.0 * kPi;
                                        // output real columns k3 whose expansion contains (s3, m3)
                                        for (int k3 = -l3; k3 <= l3; ++k3)
                                            for (int i3r = 0; i3r < n_spins; ++i3r) {
                                                if (std::abs(spins[i3r]) != std::abs(s3) || l3 < std::abs(spins[i3r]))
                                                    continue;
                                                Ent e3[2];
                                                const int n3 = column(spins[i3r], k3, e3);
                                                for (int c = 0; c < n3; ++c)
                                                    if (e3[c].s == s3 && e3[c].m == m3) {
                                                        const Cplx z = cmul(qq, Cplx{e3[c].q.re, -e3[c].q.im});
                                                        trow[static_cast<size_t>(i3r) * nbo + l3 * l3 + l3 + k3] +=
                                                            z.re * gint;
                                                    }
                                            }
                                    }
                                }
                        }
            }
}

// Block label of each slot of a row of degree L: i (L+1) + l for spin index i and
// degree l, -1 on the slots with l < |s|.
std::vector<int> slot_blocks(int L, const int* spins, int n_spins) {
    const int nb = (L + 1) * (L + 1);
    std::vector<int> out(static_cast<size_t>(n_spins) * nb, -1);
    for (int i = 0; i < n_spins; ++i)
        for (int l = std::abs(spins[i]); l <= L; ++l)
            for (int q = l * l; q < (l + 1) * (l + 1); ++q) out[static_cast<size_t>(i) * nb + q] = i * (L + 1) + l;
    return out;
}

void tensor_paths(int L1, int L2, int LO, const int* spins, int n_spins, const std::vector<double>& T,
                  std::vector<std::array<int, 3>>& paths) {
    const std::vector<int> b1 = slot_blocks(L1, spins, n_spins), b2 = slot_blocks(L2, spins, n_spins),
                           b3 = slot_blocks(LO, spins, n_spins);
    const size_t n2 = b2.size(), n3 = b3.size();
    std::set<std::array<int, 3>> seen;
    for (size_t k1 = 0; k1 < b1.size(); ++k1)
        for (size_t k2 = 0; k2 < n2; ++k2)
            for (size_t k3 = 0; k3 < n3; ++k3)
                if (std::fabs(T[(k1 * n2 + k2) * n3 + k3]) > 1e-12) seen.insert({b1[k1], b2[k2], b3[k3]});
    paths.assign(seen.begin(), seen.end());  // std::set orders lexicographically
}

void weight_paths(int L1, int L2, int LO, const int* spins, int n_spins, const std::vector<std::array<int, 3>>& paths,
                  const double* w, std::vector<double>& T) {
    const std::vector<int> b1 = slot_blocks(L1, spins, n_spins), b2 = slot_blocks(L2, spins, n_spins),
                           b3 = slot_blocks(LO, spins, n_spins);
    const size_t n2 = b2.size(), n3 = b3.size();
    std::map<std::array<int, 3>, double> weight;
    for (size_t p = 0; p < paths.size(); ++p) weight[paths[p]] = w[p];
    for (size_t k1 = 0; k1 < b1.size(); ++k1)
        for (size_t k2 = 0; k2 < n2; ++k2)
            for (size_t k3 = 0; k3 < n3; ++k3) {
                double& v = T[(k1 * n2 + k2) * n3 + k3];
                if (std::fabs(v) <= 1e-12) {
                    v = 0.0;  // quadrature round-off of an exact zero
                    continue;
                }
                v *= weight.at({b1[k1], b2[k2], b3[k3]});
            }
}

bool build_uvw_table(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags,
                     std::vector<uint32_t>& out, const std::vector<double>* dense, int role) {
    std::vector<double> own;
    if (dense == nullptr) build_dense_tensor(L1, L2, LO, spins, n_spins, flags, own);
    const std::vector<double>& T = dense != nullptr ? *dense : own;
    std::vector<std::array<int, 3>> paths;
    tensor_paths(L1, L2, LO, spins, n_spins, T, paths);
    const std::vector<int> b1 = slot_blocks(L1, spins, n_spins), b2 = slot_blocks(L2, spins, n_spins),
                           b3 = slot_blocks(LO, spins, n_spins);
    const int nc1 = static_cast<int>(b1.size()), nc2 = static_cast<int>(b2.size()), nco = static_cast<int>(b3.size());
    // tensor axes (0: x1, 1: x2, 2: out) of the role's first input, second input and output
    const int ax_a = role == 1 ? 1 : 0, ax_b = role == 0 ? 1 : 2, ax_o = role == 0 ? 2 : (role == 1 ? 0 : 1);
    const int widths[3] = {nc1, nc2, nco};
    const std::vector<int>* blk_of[3] = {&b1, &b2, &b3};
    const std::vector<int>& bo = *blk_of[ax_o];
    if (widths[ax_a] > 0xffff || widths[ax_b] > 0xffff) return false;
    std::map<std::array<int, 3>, int> index;
    for (size_t p = 0; p < paths.size(); ++p) index[paths[p]] = static_cast<int>(p);
    // first slot and width of every block of each axis; span: the role's output axis
    std::map<int, std::pair<int, int>> spans[3];
    for (int ax = 0; ax < 3; ++ax)
        for (int k = 0; k < widths[ax]; ++k) {
            const int b = (*blk_of[ax])[k];
            if (b < 0) continue;
            auto it = spans[ax].find(b);
            if (it == spans[ax].end()) spans[ax][b] = {k, 1};
            else ++it->second.second;
        }
    const std::map<int, std::pair<int, int>>& span = spans[ax_o];
    // entries per path and output component
    std::vector<std::vector<std::vector<std::pair<uint32_t, float>>>> ent(paths.size());
    for (size_t p = 0; p < paths.size(); ++p) ent[p].resize(span.at(paths[p][ax_o]).second);
    for (int k1 = 0; k1 < nc1; ++k1)
        for (int k2 = 0; k2 < nc2; ++k2)
            for (int k3 = 0; k3 < nco; ++k3) {
                const double v = T[(static_cast<size_t>(k1) * nc2 + k2) * nco + k3];
                if (std::fabs(v) <= 1e-12) continue;
                const int p = index.at({b1[k1], b2[k2], b3[k3]});
                const int k[3] = {k1, k2, k3};
                ent[p][k[ax_o] - span.at(bo[k[ax_o]]).first].push_back(
                    {static_cast<uint32_t>(k[ax_a]) | (static_cast<uint32_t>(k[ax_b]) << 16), static_cast<float>(v)});
            }
    // output blocks in slot order, each with its paths
    std::vector<int> blocks;
    for (const auto& kv : span) blocks.push_back(kv.first);
    std::vector<std::vector<int>> by_block(blocks.size());
    for (size_t p = 0; p < paths.size(); ++p)
        by_block[std::lower_bound(blocks.begin(), blocks.end(), paths[p][ax_o]) - blocks.begin()].push_back(
            static_cast<int>(p));
    std::vector<int> used;
    for (size_t b = 0; b < blocks.size(); ++b)
        if (!by_block[b].empty()) used.push_back(static_cast<int>(b));
    int max_d3 = 0;
    for (int b : used) max_d3 = std::max(max_d3, span.at(blocks[b]).second);
    const size_t rec0 = kUvwHeader + 4 * used.size();
    const size_t csr0 = rec0 + kUvwRec * paths.size();
    size_t n_csr = 0, n_ent = 0;
    for (size_t p = 0; p < paths.size(); ++p) {
        n_csr += ent[p].size() + 1;
        for (const auto& e : ent[p]) n_ent += e.size();
    }
    const size_t ent0 = csr0 + n_csr;
    out.assign(ent0 + 2 * n_ent, 0u);
    const uint32_t hdr[kUvwHeader] = {static_cast<uint32_t>(paths.size()), static_cast<uint32_t>(used.size()),
                                      static_cast<uint32_t>(widths[ax_a]), static_cast<uint32_t>(widths[ax_b]),
                                      static_cast<uint32_t>(widths[ax_o]), static_cast<uint32_t>(max_d3),
                                      static_cast<uint32_t>(rec0), static_cast<uint32_t>(ent0)};
    std::copy(hdr, hdr + kUvwHeader, out.begin());
    size_t rec = 0, csr = csr0, e_next = 0;
    for (size_t i = 0; i < used.size(); ++i) {
        const int b = used[i];
        const auto sp = span.at(blocks[b]);
        uint32_t* w = &out[kUvwHeader + 4 * i];
        w[0] = static_cast<uint32_t>(sp.first);
        w[1] = static_cast<uint32_t>(sp.second);
        w[2] = static_cast<uint32_t>(rec);
        w[3] = static_cast<uint32_t>(by_block[b].size());
        for (int p : by_block[b]) {
            uint32_t* r = &out[rec0 + kUvwRec * rec++];
            r[0] = static_cast<uint32_t>(p);
            r[1] = static_cast<uint32_t>(sp.second);
            r[2] = static_cast<uint32_t>(csr);
            for (int ax = 0; ax < 3; ++ax) {  // the path's block of x1, x2 and the output
                const auto& bs = spans[ax].at(paths[p][ax]);
                r[3 + ax] = static_cast<uint32_t>(bs.first) | (static_cast<uint32_t>(bs.second) << 16);
            }
            for (const auto& comp : ent[p]) {
                out[csr++] = static_cast<uint32_t>(e_next);
                for (const auto& e : comp) {
                    out[ent0 + 2 * e_next] = e.first;
                    std::memcpy(&out[ent0 + 2 * e_next + 1], &e.second, 4);
                    ++e_next;
                }
            }
            out[csr++] = static_cast<uint32_t>(e_next);
        }
    }
    return true;
}

void build_direct_table(int L1, int L2, int LO, const int* spins, int n_spins, unsigned flags, int role,
                        std::vector<uint32_t>& out, int* lds_floats, const std::vector<double>* dense) {
    std::vector<double> own;
    if (dense == nullptr) build_dense_tensor(L1, L2, LO, spins, n_spins, flags, own);
    const std::vector<double>& T = dense != nullptr ? *dense : own;
    const int nc1 = n_spins * (L1 + 1) * (L1 + 1), nc2 = n_spins * (L2 + 1) * (L2 + 1);
    const int nco = n_spins * (LO + 1) * (LO + 1);
    // (A, B, output) widths of the role and the index map from (a, b, o) to T
    const int na = role == 0 ? nc1 : nco, nb = role == 2 ? nc1 : nc2, no = role == 0 ? nco : (role == 1 ? nc1 : nc2);
    auto at = [&](int a, int b, int o) -> double {
        int k1 = a, k2 = b, k3 = o;  // role 0
        if (role == 1) k1 = o, k2 = b, k3 = a;
        if (role == 2) k1 = b, k2 = o, k3 = a;
        return T[(static_cast<size_t>(k1) * nc2 + k2) * nco + k3];
    };
    auto odd_stride = [](int n) { return (n % 2) ? n + 2 : n + 1; };  // odd, with a zero column at n
    const int sta = odd_stride(na), stb = odd_stride(nb), sto = odd_stride(no);
    const int hdr = 8 + 2 * (kDirectWaves + 1);  // + output and batch boundaries of the waves
    out.assign(hdr + no, 0u);
    out[0] = static_cast<uint32_t>(na);
    out[1] = static_cast<uint32_t>(nb);
    out[2] = static_cast<uint32_t>(no);
    out[3] = static_cast<uint32_t>(sta);
    out[4] = static_cast<uint32_t>(stb);
    out[5] = static_cast<uint32_t>(sto);
    out[7] = kDirectBatch;
    uint32_t nbatch = 0;
    for (int o = 0; o < no; ++o) {
        std::vector<std::pair<uint32_t, float>> ent;  // (a | b << 8, value)
        for (int a = 0; a < na; ++a)
            for (int b = 0; b < nb; ++b) {
                const double v = at(a, b, o);
                if (std::fabs(v) > 1e-12)  // the rest is quadrature round-off of exact zeros
                    ent.emplace_back(static_cast<uint32_t>(a) | (static_cast<uint32_t>(b) << 8),
                                     static_cast<float>(v));
            }
        while (ent.size() % kDirectBatch) ent.emplace_back(static_cast<uint32_t>(na) | (static_cast<uint32_t>(nb) << 8), 0.f);
        const size_t batches = ent.size() / kDirectBatch;
        out[hdr + o] = static_cast<uint32_t>(batches);
        nbatch += static_cast<uint32_t>(batches);
        for (size_t q = 0; q < batches; ++q) {
            const auto* e = &ent[q * kDirectBatch];
            for (int i = 0; i < kDirectBatch / 2; ++i) out.push_back(e[2 * i].first | (e[2 * i + 1].first << 16));
            for (int i = 0; i < kDirectBatch; ++i) {
                uint32_t bits;
                std::memcpy(&bits, &e[i].second, 4);
                out.push_back(bits);
            }
        }
    }
    out[6] = nbatch;
    out.insert(out.end(), kDirectBatch * 3, 0u);  // two zero batches that the kernel's look-ahead loads reach
    // wave w takes the whole output slots [o_w, o_(w+1)), cut where the running batch count
    // passes w+1 quarters of the total
    uint32_t seen = 0;
    int w = 1;
    out[8] = 0;
    out[8 + kDirectWaves + 1] = 0;
    for (int o = 0; o < no && w < kDirectWaves; ++o) {
        seen += out[hdr + o];
        while (w < kDirectWaves && static_cast<uint64_t>(seen) * kDirectWaves >= static_cast<uint64_t>(nbatch) * w) {
            out[8 + w] = static_cast<uint32_t>(o + 1);
            out[8 + kDirectWaves + 1 + w] = seen;
            ++w;
        }
    }
    for (; w < kDirectWaves; ++w) {  // fewer slots than waves
        out[8 + w] = static_cast<uint32_t>(no);
        out[8 + kDirectWaves + 1 + w] = nbatch;
    }
    out[8 + kDirectWaves] = static_cast<uint32_t>(no);
    out[8 + 2 * kDirectWaves + 1] = nbatch;
    *lds_floats = kDirectUnits * (sta + stb);
}

}  // namespace spingtp

namespace {

// flag bits that choose kernels, not the operation
constexpr unsigned kRouteFlags = SPINGTP_KERNEL_VALU | SPINGTP_V1_FOURIER | SPINGTP_V1_PRECONTRACT |
                                  SPINGTP_CHANNEL_WEIGHTS | SPINGTP_FULLY_CONNECTED;

spingtp_status check_args(int L1, int L2, int Lout, const int* spins, int n_spins, unsigned flags,
                          int* spin_mode) {
    if (L1 < 0 || L2 < 0 || L1 > 16 || L2 > 16 || Lout < 0 || Lout > L1 + L2) return SPINGTP_ERR_INVALID_ARG;
    if (spins == nullptr || n_spins <= 0 || n_spins > 64) return SPINGTP_ERR_INVALID_ARG;
    const unsigned basis = flags & ~kRouteFlags;
    if (basis != SPINGTP_BASIS_REAL_PAPER && basis != SPINGTP_BASIS_REAL_M0_PAIRED && basis != SPINGTP_BASIS_PARITY)
        return SPINGTP_ERR_INVALID_ARG;
    if ((flags & SPINGTP_V1_FOURIER) && (flags & SPINGTP_V1_PRECONTRACT)) return SPINGTP_ERR_INVALID_ARG;
    bool has0 = false;
    for (int i = 0; i < n_spins; ++i) {
        if (i > 0 && spins[i] <= spins[i - 1]) return SPINGTP_ERR_INVALID_ARG;
        if (spins[i] == 0) has0 = true;
        bool mirrored = false;
        for (int j = 0; j < n_spins; ++j) mirrored |= (spins[j] == -spins[i]);
        if (!mirrored) return SPINGTP_ERR_INVALID_ARG;
    }
    if (!has0) return SPINGTP_ERR_INVALID_ARG;
    if (n_spins == 1) {
        *spin_mode = 0;
    } else if (n_spins == 3 && spins[0] == -1 && spins[2] == 1) {
        *spin_mode = 1;
    } else if (n_spins == 5 && spins[0] == -2 && spins[1] == -1 && spins[3] == 1 && spins[4] == 2) {
        *spin_mode = 2;  // s_max = 2: the direct and precontracted kernels only
    } else {
        return SPINGTP_ERR_UNSUPPORTED;
    }
    return SPINGTP_OK;
}

}  // namespace

extern "C" {

const char* spingtp_status_string(spingtp_status s) {
    switch (s) {
        case SPINGTP_OK: return "ok";
        case SPINGTP_ERR_INVALID_ARG: return "invalid argument";
        case SPINGTP_ERR_UNSUPPORTED: return "unsupported configuration";
        case SPINGTP_ERR_OUT_OF_MEMORY: return "out of device memory";
        case SPINGTP_ERR_HIP: return "HIP runtime error";
        case SPINGTP_ERR_INTERNAL: return "internal error (plan self-check failed)";
        case SPINGTP_ERR_TOO_LARGE: return "request exceeds the fixed device scratch of the no-allocation entry point";
    }
    return "unknown status";
}

spingtp_status spingtp_plan_tables_host(int L1, int L2, int Lout, const int* spins, int n_spins,
                                        unsigned flags, double* tables, size_t capacity,
                                        size_t* n_tables, int* dims) {
    const bool backward = (flags & SPINGTP_TABLES_BACKWARD) != 0;
    flags &= ~SPINGTP_TABLES_BACKWARD;
    int spin_mode = 0;
    spingtp_status st = check_args(L1, L2, Lout, spins, n_spins, flags, &spin_mode);
    if (st != SPINGTP_OK) return st;
    if (n_tables == nullptr || (capacity > 0 && tables == nullptr)) return SPINGTP_ERR_INVALID_ARG;
    std::vector<double> tab;
    try {
        if (spin_mode > 1) return SPINGTP_ERR_UNSUPPORTED;
        if (!spingtp::build_tables(L1, L2, Lout, spin_mode, flags & ~kRouteFlags, tab, backward))
            return backward ? SPINGTP_ERR_UNSUPPORTED : SPINGTP_ERR_INTERNAL;
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    *n_tables = tab.size();
    const size_t n = tab.size() < capacity ? tab.size() : capacity;
    if (n) std::memcpy(tables, tab.data(), n * sizeof(double));
    if (dims) {
        const spingtp::Layout Y = spingtp::make_layout(L1, L2, Lout);
        const int d[8] = {Y.NT, Y.NP, L1, L2, Lout, n_spins, Y.pb, Y.glob};
        std::memcpy(dims, d, sizeof(d));
    }
    return SPINGTP_OK;
}

spingtp_status spingtp_dense_tensor_host(int L1, int L2, int Lout, const int* spins, int n_spins,
                                         unsigned flags, double* tensor, size_t capacity, size_t* count) {
    int spin_mode = 0;
    spingtp_status st = check_args(L1, L2, Lout, spins, n_spins, flags, &spin_mode);
    if (st != SPINGTP_OK) return st;
    if (count == nullptr || (capacity > 0 && tensor == nullptr)) return SPINGTP_ERR_INVALID_ARG;
    const size_t nc1 = static_cast<size_t>(n_spins) * (L1 + 1) * (L1 + 1);
    const size_t nc2 = static_cast<size_t>(n_spins) * (L2 + 1) * (L2 + 1);
    const size_t nco = static_cast<size_t>(n_spins) * (Lout + 1) * (Lout + 1);
    const size_t total = nc1 * nc2 * nco;
    *count = total;
    if (capacity == 0) return SPINGTP_OK;
    try {
        std::vector<double> T;
        spingtp::build_dense_tensor(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, T);
        const size_t n = total < capacity ? total : capacity;
        std::memcpy(tensor, T.data(), n * sizeof(double));
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    return SPINGTP_OK;
}

spingtp_status spingtp_mfma_operands_host(int L, uint32_t* words, size_t capacity, size_t* count) {
    if (L < 1 || L > 8 || count == nullptr || (capacity > 0 && words == nullptr)) return SPINGTP_ERR_INVALID_ARG;
    try {
        std::vector<uint32_t> w;
        spingtp::build_mfma_operands(L, w);
        *count = w.size();
        const size_t n = w.size() < capacity ? w.size() : capacity;
        if (n) std::memcpy(words, w.data(), n * sizeof(uint32_t));
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    return SPINGTP_OK;
}

spingtp_status spingtp_pre_table_host(int L1, int L2, int Lout, const int* spins, int n_spins, unsigned flags,
                                      uint32_t* words, size_t capacity, size_t* count) {
    if (count == nullptr || (capacity > 0 && words == nullptr)) return SPINGTP_ERR_INVALID_ARG;
    const bool backward = (flags & SPINGTP_TABLES_BACKWARD) != 0;
    flags &= ~SPINGTP_TABLES_BACKWARD;
    if (backward && (flags & (SPINGTP_CHANNEL_WEIGHTS | SPINGTP_FULLY_CONNECTED)) == 0 && (L1 != L2 || L2 != Lout))
        return SPINGTP_ERR_UNSUPPORTED;
    int spin_mode = 0;
    const spingtp_status st = check_args(L1, L2, Lout, spins, n_spins, flags, &spin_mode);
    if (st != SPINGTP_OK) return st;
    if (flags & SPINGTP_FULLY_CONNECTED) {  // the entry tables of the fully connected product
        try {
            std::vector<uint32_t> w;
            for (int role = backward ? 1 : 0; role < (backward ? 3 : 1); ++role) {
                std::vector<uint32_t> t;
                if (!spingtp::build_uvw_table(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, t, nullptr, role))
                    return SPINGTP_ERR_UNSUPPORTED;
                w.insert(w.end(), t.begin(), t.end());
            }
            *count = w.size();
            const size_t n = w.size() < capacity ? w.size() : capacity;
            if (n) std::memcpy(words, w.data(), n * sizeof(uint32_t));
        } catch (const std::bad_alloc&) {
            return SPINGTP_ERR_OUT_OF_MEMORY;
        }
        return SPINGTP_OK;
    }
    const bool channel_weights = (flags & SPINGTP_CHANNEL_WEIGHTS) != 0;
    if (!channel_weights && spingtp::find_pre_kernel(L1, L2, Lout, n_spins, 0) == nullptr)
        return SPINGTP_ERR_UNSUPPORTED;
    try {
        std::vector<uint32_t> w;
        if (channel_weights && backward) {  // the entry lists of spingtp_backward_v1_weighted
            if (!spingtp::build_bwd_v1w_table(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, w, nullptr))
                return SPINGTP_ERR_UNSUPPORTED;
        } else if (channel_weights) {  // the table of spingtp_forward_v1_weighted, as a plan with the flag builds it
            const int nc1 = n_spins * (L1 + 1) * (L1 + 1), nc2 = n_spins * (L2 + 1) * (L2 + 1);
            const int nco = n_spins * (Lout + 1) * (Lout + 1);
            int rows = 0, ks = 0, nt = 0;
            (void)spingtp::build_pre_tables_channel_weighted(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, 0, w,
                                                             &rows);
            if (nc2 > spingtp::kPreMaxNC ||
                spingtp::find_pre_weighted_kernel((std::max(rows, nc1) + 15) / 16, (nco + 15) / 16, 0, &ks, &nt) ==
                    nullptr ||
                !spingtp::build_pre_tables_channel_weighted(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, ks, w,
                                                            &rows))
                return SPINGTP_ERR_UNSUPPORTED;
        } else if (!spingtp::build_pre_tables(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, w, backward)) {
            return SPINGTP_ERR_UNSUPPORTED;
        }
        *count = w.size();
        const size_t n = w.size() < capacity ? w.size() : capacity;
        if (n) std::memcpy(words, w.data(), n * sizeof(uint32_t));
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    return SPINGTP_OK;
}

spingtp_status spingtp_direct_table_host(int L1, int L2, int Lout, const int* spins, int n_spins, unsigned flags,
                                         int role, uint32_t* words, size_t capacity, size_t* count) {
    if (count == nullptr || (capacity > 0 && words == nullptr) || role < 0 || role > 2) return SPINGTP_ERR_INVALID_ARG;
    int spin_mode = 0;
    const spingtp_status st = check_args(L1, L2, Lout, spins, n_spins, flags, &spin_mode);
    if (st != SPINGTP_OK) return st;
    try {
        std::vector<uint32_t> w;
        int lds_floats = 0;
        const int nmax = n_spins * (std::max(L1, std::max(L2, Lout)) + 1) * (std::max(L1, std::max(L2, Lout)) + 1);
        if (nmax > spingtp::kDirectMaxRow) return SPINGTP_ERR_UNSUPPORTED;
        spingtp::build_direct_table(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, role, w, &lds_floats);
        if (spingtp::find_direct_kernel(lds_floats, 0) == nullptr) return SPINGTP_ERR_UNSUPPORTED;
        *count = w.size();
        const size_t n = w.size() < capacity ? w.size() : capacity;
        if (n) std::memcpy(words, w.data(), n * sizeof(uint32_t));
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    return SPINGTP_OK;
}

spingtp_status spingtp_conj_map_host(int L, const int* spins, int n_spins, unsigned flags, uint32_t* words,
                                     size_t capacity, size_t* count) {
    if (count == nullptr || (capacity > 0 && words == nullptr)) return SPINGTP_ERR_INVALID_ARG;
    int spin_mode = 0;
    const spingtp_status st = check_args(L, L, L, spins, n_spins, flags, &spin_mode);
    if (st != SPINGTP_OK) return st;
    try {
        std::vector<uint32_t> w;
        if (!spingtp::build_conj_map(L, spins, n_spins, flags & ~kRouteFlags, w)) return SPINGTP_ERR_INTERNAL;
        *count = w.size();
        const size_t n = w.size() < capacity ? w.size() : capacity;
        if (n) std::memcpy(words, w.data(), n * sizeof(uint32_t));
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    return SPINGTP_OK;
}

namespace {

// Everything a plan holds, built on the host: the chosen kernels and the float64 /
// word tables that go to the device.
struct PlanHost {
    int spin_mode = 0, dir_lds = 0;
    const spingtp::KernelEntry *k = nullptr, *kd = nullptr, *kv1 = nullptr, *kw = nullptr;
    std::vector<double> tab, tab_bwd;
    std::vector<uint32_t> aux, pre, pre_bwd, dir, dir_b1, dir_b2, pre_w, bw1w, uvw;
    size_t uvw_off[3] = {0, 0, 0};  // first word of each role's table in uvw
    bool padded = false;            // mixed degrees on the large-degree kernel (aux: 3 degree triples)
    spingtp::Bw1wShape bw1w_shape{};
    bool has_backward = false, same_bwd = false;
};

// weights: one per path of spingtp_paths_host (n_weights of them), or nullptr for the
// unweighted product.
spingtp_status build_plan_host(int L1, int L2, int Lout, const int* spins, int n_spins, spingtp_dtype dtype,
                               unsigned flags, const double* weights, size_t n_weights, PlanHost& h) {
    int spin_mode = 0;
    spingtp_status st = check_args(L1, L2, Lout, spins, n_spins, flags, &spin_mode);
    if (st != SPINGTP_OK) return st;
    if (dtype != SPINGTP_FP32 && dtype != SPINGTP_BF16) return SPINGTP_ERR_INVALID_ARG;
    const bool weighted = weights != nullptr;
    // weighted plans: the Fourier route computes the unweighted sum over all paths at once
    if (weighted && (flags & SPINGTP_V1_FOURIER)) return SPINGTP_ERR_UNSUPPORTED;
    // per-channel path weights are given at each call; not combined with plan-level ones
    const bool channel_weights = (flags & SPINGTP_CHANNEL_WEIGHTS) != 0;
    if (channel_weights && weighted) return SPINGTP_ERR_INVALID_ARG;
    const spingtp::KernelEntry* k = nullptr;
    if ((flags & SPINGTP_KERNEL_VALU) == 0 && !weighted)
        k = spingtp::find_mfma_kernel(L1, L2, Lout, spin_mode, static_cast<int>(dtype));
    const bool parity_tiles = spin_mode == 1 && (flags & ~kRouteFlags) == SPINGTP_BASIS_PARITY;
    if (k == nullptr && !weighted)
        k = spingtp::find_kernel(L1, L2, Lout, spin_mode, static_cast<int>(dtype), parity_tiles);
    // the direct kernel: shapes without a Fourier kernel, and the gradients of shapes
    // whose transposed degrees have none, where its LDS tile fits
    auto odd_stride = [](int n) { return (n % 2) ? n + 2 : n + 1; };
    const int bsz = (L1 + 1) * (L1 + 1), bsz2 = (L2 + 1) * (L2 + 1), bszo = (Lout + 1) * (Lout + 1);
    // (the LDS holds two of the three rows; every role pairs a different two, so size for the largest pair,
    // and the entry indices are 8-bit)
    const int r1 = odd_stride(n_spins * bsz), r2 = odd_stride(n_spins * bsz2), ro = odd_stride(n_spins * bszo);
    const int dir_lds = spingtp::kDirectUnits * (r1 + r2 + ro - std::min(r1, std::min(r2, ro)));
    const bool dir_idx_ok = n_spins * std::max(bsz, std::max(bsz2, bszo)) <= spingtp::kDirectMaxRow;
    const spingtp::KernelEntry* kd = dir_idx_ok ? spingtp::find_direct_kernel(dir_lds, static_cast<int>(dtype)) : nullptr;
    const bool fourier_bwd = k != nullptr && L1 == L2 && L2 == Lout;
    if (k == nullptr) k = kd;
    // mixed degrees whose rows exceed the direct kernel's: the large-degree kernel of the
    // largest degree, with x1 and x2 padded by zeros as it stages them and the product
    // truncated to Lout as it stores it (exact: its grid integrates degree 3 max(L1, L2,
    // Lout) >= L1 + L2 + Lout); the three degrees reach it through the plan's aux words.
    // Forward and V = 1 only.
    int L_pad = -1;
    if (k == nullptr && !weighted && spin_mode < 2) {
        const int Lm = std::max(L1, std::max(L2, Lout));
        const spingtp::KernelEntry* kb =
            spingtp::find_kernel(Lm, Lm, Lm, spin_mode, static_cast<int>(dtype), parity_tiles);
        if (kb != nullptr && kb->family == 3)
            kb = spingtp::find_big_padded_kernel(Lm, spin_mode, static_cast<int>(dtype), parity_tiles);
        if (kb != nullptr && kb->family == 3) {
            k = kb;
            L_pad = Lm;
        }
    }
    h.padded = L_pad >= 0;
    const spingtp::KernelEntry* kv1 = nullptr;
    if ((flags & SPINGTP_V1_FOURIER) == 0) {
        kv1 = spingtp::find_pre_kernel(L1, L2, Lout, n_spins, static_cast<int>(dtype));
        // measured crossover: with rows longer than 75 slots (degree 5 with spins {-1, 0, 1}:
        // 0.54 against 0.66 ms at 8192 edges x 128 channels) the Fourier route is faster
        const int rows = n_spins * (std::max(L1, Lout) + 1) * (std::max(L1, Lout) + 1);
        if (kv1 != nullptr && k != nullptr && k->family != 6 && rows > 75 && (flags & SPINGTP_V1_PRECONTRACT) == 0)
            kv1 = nullptr;
        if (kv1 == nullptr && (flags & SPINGTP_V1_PRECONTRACT)) return SPINGTP_ERR_UNSUPPORTED;
    }
    if (kv1 == nullptr) kv1 = k;
    if (kv1 == nullptr) return SPINGTP_ERR_UNSUPPORTED;
    const unsigned basis = flags & ~kRouteFlags;

    std::vector<double>& tab = h.tab;
    std::vector<double>& tab_bwd = h.tab_bwd;
    std::vector<uint32_t>&aux = h.aux, &pre = h.pre, &pre_bwd = h.pre_bwd, &dir = h.dir, &dir_b1 = h.dir_b1,
                         &dir_b2 = h.dir_b2, &pre_w = h.pre_w, &bw1w = h.bw1w;
    spingtp::Bw1wShape& bw1w_shape = h.bw1w_shape;
    const spingtp::KernelEntry*& kw = h.kw;
    bool &has_backward = h.has_backward, &same_bwd = h.same_bwd;
    h.spin_mode = spin_mode;
    h.dir_lds = dir_lds;
    h.k = k;
    h.kd = kd;
    h.kv1 = kv1;
    try {
        if (L_pad >= 0) {  // the tables of the padded degree, and the true degrees
            if (!spingtp::build_tables(L_pad, L_pad, L_pad, spin_mode, basis, tab)) return SPINGTP_ERR_INTERNAL;
            // (x1, x2 -> out) of the forward, then the gradient launches' (grad_out, x2 -> grad_x1)
            // and (grad_out, x1 -> grad_x2)
            const uint32_t a = static_cast<uint32_t>(L1), b = static_cast<uint32_t>(L2),
                           c = static_cast<uint32_t>(Lout);
            aux = {a, b, c, c, b, a, c, a, b};
            // the gradients: the degree-L ones of the padded functions, truncated
            if (spingtp::build_tables(L_pad, L_pad, L_pad, spin_mode, basis, tab_bwd, true)) {
                has_backward = true;
                same_bwd = tab_bwd == tab;
            }
        } else if (spin_mode < 2 && !weighted && !spingtp::build_tables(L1, L2, Lout, spin_mode, basis, tab)) {
            return SPINGTP_ERR_INTERNAL;
        }
        int lds_floats = 0;
        std::vector<double> dense;  // built once for the direct kernel's tables (and weighted plans)
        if ((k != nullptr && k->family == 6) || (kd != nullptr && !fourier_bwd) || weighted)
            spingtp::build_dense_tensor(L1, L2, Lout, spins, n_spins, basis, dense);
        if (weighted) {
            std::vector<std::array<int, 3>> paths;
            spingtp::tensor_paths(L1, L2, Lout, spins, n_spins, dense, paths);
            if (n_weights != paths.size()) return SPINGTP_ERR_INVALID_ARG;
            for (size_t i = 0; i < n_weights; ++i)
                if (!std::isfinite(weights[i])) return SPINGTP_ERR_INVALID_ARG;
            spingtp::weight_paths(L1, L2, Lout, spins, n_spins, paths, weights, dense);
        }
        if (k != nullptr && k->family == 6)
            spingtp::build_direct_table(L1, L2, Lout, spins, n_spins, basis, 0, dir, &lds_floats, &dense);
        if (channel_weights) {  // path slots first, then the instantiation that holds them
            const int nc2 = n_spins * (L2 + 1) * (L2 + 1), nco = n_spins * (Lout + 1) * (Lout + 1);
            const int nc1 = n_spins * (L1 + 1) * (L1 + 1);
            int rows = 0, ks = 0, nt = 0;
            if (nc2 <= spingtp::kPreMaxNC) {
                // with ks = 0 the builder only counts the path slots
                (void)spingtp::build_pre_tables_channel_weighted(L1, L2, Lout, spins, n_spins, basis, 0, pre_w,
                                                                 &rows);
                kw = spingtp::find_pre_weighted_kernel((std::max(rows, nc1) + 15) / 16, (nco + 15) / 16,
                                                       static_cast<int>(dtype), &ks, &nt);
            }
            if (kw == nullptr ||
                !spingtp::build_pre_tables_channel_weighted(L1, L2, Lout, spins, n_spins, basis, ks, pre_w, &rows)) {
                kw = nullptr;
                pre_w.clear();
            }
            // the gradients (spingtp_backward_v1_weighted) where their tiles fit; a plan
            // needs the forward or the gradients
            if (!spingtp::build_bwd_v1w_table(L1, L2, Lout, spins, n_spins, basis, bw1w, &bw1w_shape))
                bw1w.clear();
            if (pre_w.empty() && bw1w.empty()) return SPINGTP_ERR_UNSUPPORTED;
        }
        if (kd != nullptr && !fourier_bwd) {
            spingtp::build_direct_table(L1, L2, Lout, spins, n_spins, basis, 1, dir_b1, &lds_floats, &dense);
            spingtp::build_direct_table(L1, L2, Lout, spins, n_spins, basis, 2, dir_b2, &lds_floats, &dense);
        }
        if (k != nullptr && k->family == 4) spingtp::build_mfma_operands(L1, aux);
        if (flags & SPINGTP_FULLY_CONNECTED) {
            // the forward's table, then those of the gradients w.r.t. x1 and x2, in one buffer
            for (int role = 0; role < 3; ++role) {
                std::vector<uint32_t> t;
                if (!spingtp::build_uvw_table(L1, L2, Lout, spins, n_spins, basis, t, dense.empty() ? nullptr : &dense,
                                              role))
                    return SPINGTP_ERR_UNSUPPORTED;
                h.uvw_off[role] = h.uvw.size();
                h.uvw.insert(h.uvw.end(), t.begin(), t.end());
            }
        }
        if (kv1->family == 5 &&
            !spingtp::build_pre_tables(L1, L2, Lout, spins, n_spins, basis, pre, false, weighted ? &dense : nullptr))
            return SPINGTP_ERR_INTERNAL;
        // spingtp_backward_v1 on the precontracted kernel: the same table with J x2 (the
        // conjugation identity holds for the unweighted tensor only)
        if (kv1->family == 5 && L1 == L2 && L2 == Lout && !weighted &&
            !spingtp::build_pre_tables(L1, L2, Lout, spins, n_spins, basis, pre_bwd, true))
            pre_bwd.clear();
        // spingtp_backward: square plans with a forward kernel, input 2 conjugated
        if (fourier_bwd && spingtp::build_tables(L1, L2, Lout, spin_mode, basis, tab_bwd, true)) {
            has_backward = true;
            same_bwd = tab_bwd == tab;
        }
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    return SPINGTP_OK;
}

// Device functions of the upload; plan creation passes HIP's, the host self-test its own.
struct DeviceApi {
    void* ctx;
    int (*alloc)(void* ctx, void** p, size_t bytes);  // 0 ok, 1 out of memory, 2 other failure
    int (*copy)(void* ctx, void* dst, const void* src, size_t bytes);
    void (*release)(void* ctx, void* p);
};

// The device copies of a plan's tables; all null before a successful upload.
struct PlanDevice {
    float *tab = nullptr, *tab_bwd = nullptr;
    uint32_t *aux = nullptr, *pre = nullptr, *pre_bwd = nullptr, *dir = nullptr, *dir_b1 = nullptr,
             *dir_b2 = nullptr, *pre_w = nullptr, *bw1w = nullptr, *uvw = nullptr;
};

// Uploads every non-empty table (fp32 tables rounded to nearest).  On any failure every
// buffer allocated so far is released and d is left all null: nothing leaks.
spingtp_status upload_plan(const PlanHost& h, const DeviceApi& api, PlanDevice& d) {
    d = PlanDevice{};
    std::vector<void*> held;
    int fail = 0;
    auto put = [&](const void* src, size_t bytes, void** dst) {
        if (fail != 0 || bytes == 0) return;
        void* p = nullptr;
        fail = api.alloc(api.ctx, &p, bytes);
        if (fail != 0) return;
        held.push_back(p);
        if (api.copy(api.ctx, p, src, bytes) != 0) fail = 2;
        *dst = p;
    };
    try {
        std::vector<float> f(h.tab.size());
        for (size_t i = 0; i < f.size(); ++i) f[i] = static_cast<float>(h.tab[i]);
        put(f.data(), f.size() * sizeof(float), reinterpret_cast<void**>(&d.tab));
        if (h.has_backward && !h.same_bwd) {
            f.assign(h.tab_bwd.size(), 0.f);
            for (size_t i = 0; i < f.size(); ++i) f[i] = static_cast<float>(h.tab_bwd[i]);
            put(f.data(), f.size() * sizeof(float), reinterpret_cast<void**>(&d.tab_bwd));
        }
    } catch (const std::bad_alloc&) {
        fail = 1;
    }
    const std::pair<const std::vector<uint32_t>*, uint32_t**> words[] = {
        {&h.aux, &d.aux}, {&h.pre, &d.pre}, {&h.pre_bwd, &d.pre_bwd}, {&h.dir, &d.dir}, {&h.dir_b1, &d.dir_b1},
        {&h.dir_b2, &d.dir_b2}, {&h.pre_w, &d.pre_w}, {&h.bw1w, &d.bw1w}, {&h.uvw, &d.uvw}};
    for (const auto& w : words)
        put(w.first->data(), w.first->size() * sizeof(uint32_t), reinterpret_cast<void**>(w.second));
    if (fail == 0) return SPINGTP_OK;
    for (void* p : held) api.release(api.ctx, p);
    d = PlanDevice{};
    return fail == 1 ? SPINGTP_ERR_OUT_OF_MEMORY : SPINGTP_ERR_HIP;
}

int hip_alloc(void*, void** p, size_t bytes) {
    const hipError_t e = hipMalloc(p, bytes);
    return e == hipSuccess ? 0 : (e == hipErrorOutOfMemory ? 1 : 2);
}
int hip_copy(void*, void* dst, const void* src, size_t bytes) {
    return hipMemcpy(dst, src, bytes, hipMemcpyHostToDevice) == hipSuccess ? 0 : 2;
}
void hip_release(void*, void* p) {
    (void)hipFree(p);
}

}  // namespace

static spingtp_status create_plan(int L1, int L2, int Lout, const int* spins, int n_spins, spingtp_dtype dtype,
                                  unsigned flags, const double* weights, size_t n_weights, spingtp_plan* out_plan) {
    if (out_plan == nullptr) return SPINGTP_ERR_INVALID_ARG;
    *out_plan = nullptr;
    PlanHost h;
    const spingtp_status st = build_plan_host(L1, L2, Lout, spins, n_spins, dtype, flags, weights, n_weights, h);
    if (st != SPINGTP_OK) return st;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return SPINGTP_ERR_HIP;
    PlanDevice d;
    const DeviceApi api{nullptr, hip_alloc, hip_copy, hip_release};
    const spingtp_status su = upload_plan(h, api, d);
    if (su != SPINGTP_OK) return su;
    spingtp_plan p = new (std::nothrow) spingtp_plan_s;
    if (p == nullptr) {
        for (void* q : {static_cast<void*>(d.tab), static_cast<void*>(d.tab_bwd), static_cast<void*>(d.aux),
                        static_cast<void*>(d.pre), static_cast<void*>(d.pre_bwd), static_cast<void*>(d.dir),
                        static_cast<void*>(d.dir_b1), static_cast<void*>(d.dir_b2), static_cast<void*>(d.pre_w),
                        static_cast<void*>(d.bw1w), static_cast<void*>(d.uvw)})
            if (q != nullptr) (void)hipFree(q);
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    p->L1 = L1;
    p->L2 = L2;
    p->LO = Lout;
    p->spin_mode = h.spin_mode;
    p->n_spins = n_spins;
    p->dtype = dtype;
    p->flags = flags;
    p->device = dev;
    p->d_tab = d.tab;
    p->n_tab = h.tab.size();
    p->d_aux = d.aux;
    p->d_pre = d.pre;
    p->d_pre_bwd = d.pre_bwd;
    p->d_tab_bwd = h.has_backward ? (h.same_bwd ? d.tab : d.tab_bwd) : nullptr;
    p->own_tab_bwd = d.tab_bwd != nullptr;
    p->d_dir = d.dir;
    p->d_dir_b1 = d.dir_b1;
    p->d_dir_b2 = d.dir_b2;
    p->kernel_dir = d.dir_b1 != nullptr ? h.kd : nullptr;
    p->dir_lds_floats = h.dir_lds;
    p->d_pre_w = d.pre_w;
    p->kernel_v1w = d.pre_w != nullptr ? h.kw : nullptr;
    p->d_bw1w = d.bw1w;
    p->bw1w = h.bw1w_shape;
    p->d_uvw = d.uvw;
    for (int role = 0; role < 3; ++role) {
        const size_t o = h.uvw_off[role];
        p->uvw_off[role] = o;
        p->uvw_blocks[role] = h.uvw.empty() ? 0 : static_cast<int>(h.uvw[o + 1]);
        p->uvw_max_d3[role] = h.uvw.empty() ? 0 : static_cast<int>(h.uvw[o + 5]);
    }
    p->uvw_paths = h.uvw.empty() ? 0 : static_cast<int>(h.uvw[0]);
    p->kernel = h.k;
    p->kernel_v1 = h.kv1;
    p->padded = h.padded;
    *out_plan = p;
    return SPINGTP_OK;
}


extern "C" spingtp_status spingtp_plan_upload_selftest_host(int L1, int L2, int Lout, const int* spins, int n_spins,
                                                            spingtp_dtype dtype, unsigned flags, int fail_at,
                                                            int* n_allocs, int* n_live) {
    if (n_allocs == nullptr || n_live == nullptr) return SPINGTP_ERR_INVALID_ARG;
    PlanHost h;
    const spingtp_status st = build_plan_host(L1, L2, Lout, spins, n_spins, dtype, flags, nullptr, 0, h);
    if (st != SPINGTP_OK) return st;
    struct Counter {
        int fail_at, allocs = 0, live = 0;
    } c{fail_at};
    const DeviceApi api{&c,
                        [](void* ctx, void** p, size_t bytes) -> int {
                            Counter& k = *static_cast<Counter*>(ctx);
                            if (k.allocs++ == k.fail_at) return 1;
                            *p = std::malloc(bytes);
                            if (*p == nullptr) return 1;
                            ++k.live;
                            return 0;
                        },
                        [](void*, void* dst, const void* src, size_t bytes) -> int {
                            std::memcpy(dst, src, bytes);
                            return 0;
                        },
                        [](void* ctx, void* p) {
                            --static_cast<Counter*>(ctx)->live;
                            std::free(p);
                        }};
    PlanDevice d;
    const spingtp_status su = upload_plan(h, api, d);
    *n_allocs = c.allocs;
    *n_live = c.live;
    if (su == SPINGTP_OK)
        for (void* q : {static_cast<void*>(d.tab), static_cast<void*>(d.tab_bwd), static_cast<void*>(d.aux),
                        static_cast<void*>(d.pre), static_cast<void*>(d.pre_bwd), static_cast<void*>(d.dir),
                        static_cast<void*>(d.dir_b1), static_cast<void*>(d.dir_b2), static_cast<void*>(d.pre_w),
                        static_cast<void*>(d.bw1w), static_cast<void*>(d.uvw)})
            if (q != nullptr) api.release(api.ctx, q);
    return su;
}

spingtp_status spingtp_plan_create(int L1, int L2, int Lout, const int* spins, int n_spins,
                                   spingtp_dtype dtype, unsigned flags, spingtp_plan* out_plan) {
    return create_plan(L1, L2, Lout, spins, n_spins, dtype, flags, nullptr, 0, out_plan);
}

spingtp_status spingtp_plan_create_weighted(int L1, int L2, int Lout, const int* spins, int n_spins,
                                            spingtp_dtype dtype, unsigned flags, const double* weights,
                                            size_t n_weights, spingtp_plan* out_plan) {
    if (weights == nullptr) {
        if (out_plan != nullptr) *out_plan = nullptr;
        return SPINGTP_ERR_INVALID_ARG;
    }
    return create_plan(L1, L2, Lout, spins, n_spins, dtype, flags, weights, n_weights, out_plan);
}

spingtp_status spingtp_paths_host(int L1, int L2, int Lout, const int* spins, int n_spins, unsigned flags,
                                  int* triples, size_t capacity, size_t* count) {
    if (count == nullptr || (capacity > 0 && triples == nullptr)) return SPINGTP_ERR_INVALID_ARG;
    int spin_mode = 0;
    const spingtp_status st = check_args(L1, L2, Lout, spins, n_spins, flags, &spin_mode);
    if (st != SPINGTP_OK) return st;
    try {
        std::vector<double> T;
        spingtp::build_dense_tensor(L1, L2, Lout, spins, n_spins, flags & ~kRouteFlags, T);
        std::vector<std::array<int, 3>> paths;
        spingtp::tensor_paths(L1, L2, Lout, spins, n_spins, T, paths);
        *count = paths.size();
        const size_t n = paths.size() < capacity ? paths.size() : capacity;
        for (size_t i = 0; i < n; ++i)
            for (int j = 0; j < 3; ++j) triples[3 * i + j] = paths[i][j];
    } catch (const std::bad_alloc&) {
        return SPINGTP_ERR_OUT_OF_MEMORY;
    }
    return SPINGTP_OK;
}

spingtp_status spingtp_plan_destroy(spingtp_plan plan) {
    if (plan == nullptr) return SPINGTP_OK;
    int cur = 0;
    hipError_t first = hipGetDevice(&cur);
    const bool switched = first == hipSuccess && cur != plan->device;
    if (switched) first = hipSetDevice(plan->device);
    // every buffer is freed even after a failure; the first error is reported
    auto release = [&first](void* p) {
        if (p == nullptr) return;
        const hipError_t e = hipFree(p);
        if (first == hipSuccess) first = e;
    };
    release(plan->d_tab);
    release(plan->d_aux);
    release(plan->d_dir);
    release(plan->d_dir_b1);
    release(plan->d_dir_b2);
    release(plan->d_pre_w);
    release(plan->d_bw1w);
    release(plan->d_pre);
    release(plan->d_pre_bwd);
    release(plan->d_uvw);
    if (plan->own_tab_bwd) release(plan->d_tab_bwd);
    if (switched) (void)hipSetDevice(cur);
    delete plan;
    return first == hipSuccess ? SPINGTP_OK : SPINGTP_ERR_HIP;
}

spingtp_status spingtp_plan_kernel_info(spingtp_plan plan, int* info) {
    if (plan == nullptr || info == nullptr) return SPINGTP_ERR_INVALID_ARG;
    if (plan->kernel == nullptr) return SPINGTP_ERR_UNSUPPORTED;
    info[0] = plan->kernel->waves;
    info[1] = plan->kernel->units;
    info[2] = plan->kernel->family == 6 ? plan->dir_lds_floats * 4 : plan->kernel->lds_bytes;
    info[3] = plan->kernel->family;
    return SPINGTP_OK;
}

spingtp_status spingtp_plan_kernel_info_v1(spingtp_plan plan, int* info) {
    if (plan == nullptr || info == nullptr) return SPINGTP_ERR_INVALID_ARG;
    info[0] = plan->kernel_v1->waves;
    info[1] = plan->kernel_v1->units;
    info[2] = plan->kernel_v1->family == 6 ? plan->dir_lds_floats * 4 : plan->kernel_v1->lds_bytes;
    info[3] = plan->kernel_v1->family;
    return SPINGTP_OK;
}

}  // extern "C"
