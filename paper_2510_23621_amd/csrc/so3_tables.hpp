// Host-side SO(3) tables for the MACE layer: real Clebsch-Gordan couplings
// (edge product of Eq. 26, and the coupling trees of Eq. 27) and the
// selection of coupling trees that form the generalised-CG basis of the
// symmetric contraction.
//
// Conventions (fixed by this library; the paper names the objects only):
//  * real harmonics: m = -l..l, m>0 ~ cos(m phi), m<0 ~ sin(|m| phi), no
//    Condon-Shortley phase, sum_m Y_lm^2 = 2l+1 (so Y_1 = sqrt3 (y, z, x));
//  * real CG C^{l3}_{l1 l2}[m1][m2][m3]: the complex (Condon-Shortley) CG
//    from the Racah formula, carried to the real basis by the unitary
//    complex->real change of basis, made real by removing a global phase,
//    with the first nonzero entry (lexicographic m1, m2, m3) positive.
//    Orthonormal: sum_{m1 m2} C[m1][m2][m3] C[m1][m2][m3'] = delta.
//  * coupling trees over A = 0e+1o+2e+3o (16 components, block l at l*l):
//      nu=1 (l1), l1 = L;  nu=2 (l1<=l2);  nu=3 (l1<=l2<=l3; l12 ascending),
//    parity (-1)^(sum l) = parity of L; each tree symmetrised over its nu
//    factors, kept when linearly independent of the trees kept before it
//    (modified Gram-Schmidt, relative residual > 1e-8), with scale 1/||Sym T||.
//
// Header-only, double precision, no dependencies beyond the C++ library.
#pragma once

#include <algorithm>
#include <array>
#include <cmath>
#include <complex>
#include <cstdint>
#include <map>
#include <stdexcept>
#include <tuple>
#include <vector>

namespace so3h {

using cd = std::complex<double>;

inline double fact(int n) {
  if (n < 0) throw std::runtime_error("negative factorial");
  double r = 1.0;
  for (int i = 2; i <= n; ++i) r *= i;
  return r;
}

// <j1 m1 j2 m2 | J M>, Racah's closed form (Condon-Shortley phase).
inline double cg_complex(int j1, int m1, int j2, int m2, int J, int M) {
  if (M != m1 + m2) return 0.0;
  if (J < std::abs(j1 - j2) || J > j1 + j2) return 0.0;
  if (std::abs(m1) > j1 || std::abs(m2) > j2 || std::abs(M) > J) return 0.0;
  double pre = std::sqrt((2.0 * J + 1.0) * fact(J + j1 - j2) * fact(J - j1 + j2) * fact(j1 + j2 - J) /
                         fact(j1 + j2 + J + 1));
  pre *= std::sqrt(fact(J + M) * fact(J - M) * fact(j1 - m1) * fact(j1 + m1) * fact(j2 - m2) * fact(j2 + m2));
  double s = 0.0;
  for (int k = 0; k <= j1 + j2 + J; ++k) {
    int a1 = j1 + j2 - J - k, a2 = j1 - m1 - k, a3 = j2 + m2 - k, a4 = J - j2 + m1 + k, a5 = J - j1 - m2 + k;
    if (a1 < 0 || a2 < 0 || a3 < 0 || a4 < 0 || a5 < 0) continue;
    double t = 1.0 / (fact(k) * fact(a1) * fact(a2) * fact(a3) * fact(a4) * fact(a5));
    s += (k % 2 ? -t : t);
  }
  return pre * s;
}

// Q[m+l][mu+l]: real harmonic m = sum_mu Q[m][mu] * complex harmonic mu.
inline std::vector<cd> complex_to_real(int l) {
  int n = 2 * l + 1;
  std::vector<cd> Q(n * n, cd(0, 0));
  const double h = 1.0 / std::sqrt(2.0);
  for (int m = -l; m <= l; ++m) {
    int i = m + l;
    if (m == 0) {
      Q[i * n + l] = 1.0;
    } else if (m > 0) {
      Q[i * n + (l - m)] = h;
      Q[i * n + (l + m)] = (m % 2 ? -h : h);
    } else {
      int mu = -m;
      Q[i * n + (l - mu)] = cd(0, h);
      Q[i * n + (l + mu)] = cd(0, (mu % 2 ? h : -h));
    }
  }
  return Q;
}

struct CGTensor {
  int l1 = 0, l2 = 0, l3 = 0;
  std::vector<double> v;   // [(2l1+1)][(2l2+1)][(2l3+1)]
  double at(int m1, int m2, int m3) const {
    return v[((m1) * (2 * l2 + 1) + m2) * (2 * l3 + 1) + m3];
  }
};

inline CGTensor real_cg(int l1, int l2, int l3) {
  if (l3 < std::abs(l1 - l2) || l3 > l1 + l2) throw std::runtime_error("triangle");
  int n1 = 2 * l1 + 1, n2 = 2 * l2 + 1, n3 = 2 * l3 + 1;
  auto Q1 = complex_to_real(l1), Q2 = complex_to_real(l2), Q3 = complex_to_real(l3);
  std::vector<cd> c(n1 * n2 * n3, cd(0, 0));
  for (int a = 0; a < n1; ++a)
    for (int b = 0; b < n2; ++b)
      for (int d = 0; d < n3; ++d) {
        cd acc(0, 0);
        for (int u1 = 0; u1 < n1; ++u1) {
          cd q1 = std::conj(Q1[a * n1 + u1]);
          if (q1 == cd(0, 0)) continue;
          for (int u2 = 0; u2 < n2; ++u2) {
            cd q2 = std::conj(Q2[b * n2 + u2]);
            if (q2 == cd(0, 0)) continue;
            int mu3 = (u1 - l1) + (u2 - l2);
            if (std::abs(mu3) > l3) continue;
            cd q3 = Q3[d * n3 + (mu3 + l3)];
            if (q3 == cd(0, 0)) continue;
            acc += q1 * q2 * q3 * cg_complex(l1, u1 - l1, l2, u2 - l2, l3, mu3);
          }
        }
        c[(a * n2 + b) * n3 + d] = acc;
      }
  // remove the global phase using the largest entry
  size_t kmax = 0;
  for (size_t i = 1; i < c.size(); ++i)
    if (std::abs(c[i]) > std::abs(c[kmax])) kmax = i;
  cd ph = c[kmax] / std::abs(c[kmax]);
  CGTensor t;
  t.l1 = l1; t.l2 = l2; t.l3 = l3;
  t.v.resize(c.size());
  for (size_t i = 0; i < c.size(); ++i) {
    cd z = c[i] / ph;
    if (std::abs(z.imag()) > 1e-10) throw std::runtime_error("real CG has imaginary part");
    double r = z.real();
    t.v[i] = std::abs(r) < 1e-12 ? 0.0 : r;
  }
  for (size_t i = 0; i < t.v.size(); ++i) {
    if (std::abs(t.v[i]) > 1e-9) {
      if (t.v[i] < 0)
        for (auto& x : t.v) x = -x;
      break;
    }
  }
  return t;
}

// ---------------------------------------------------------------------------
// coupling trees of the symmetric contraction
// ---------------------------------------------------------------------------
constexpr int kAL = 3;                    // A carries l = 0..3
constexpr int kAC = (kAL + 1) * (kAL + 1);  // 16 components

struct Tree {
  int nu = 1;
  int l1 = 0, l2 = 0, l3 = 0, l12 = 0;    // unused entries 0
  double scale = 1.0;                     // 1 / ||Sym T||_F
};

inline std::vector<Tree> candidate_trees(int nu, int L, int parity) {
  std::vector<Tree> out;
  auto par = [](int s) { return (s % 2) ? -1 : 1; };
  if (nu == 1) {
    for (int a = 0; a <= kAL; ++a)
      if (a == L && par(a) == parity) out.push_back(Tree{1, a, 0, 0, 0, 1.0});
  } else if (nu == 2) {
    for (int a = 0; a <= kAL; ++a)
      for (int b = 0; b <= kAL; ++b)
        if (a <= b && std::abs(a - b) <= L && L <= a + b && par(a + b) == parity)
          out.push_back(Tree{2, a, b, 0, 0, 1.0});
  } else if (nu == 3) {
    for (int a = 0; a <= kAL; ++a)
      for (int b = 0; b <= kAL; ++b)
        for (int c = 0; c <= kAL; ++c) {
          if (!(a <= b && b <= c) || par(a + b + c) != parity) continue;
          for (int l12 = std::abs(a - b); l12 <= a + b; ++l12)
            if (std::abs(l12 - c) <= L && L <= l12 + c) out.push_back(Tree{3, a, b, c, l12, 1.0});
        }
  }
  return out;
}

// Dense symmetrised tensor S[M][a1..a_nu] (flattened, a-index fastest).
inline std::vector<double> symmetrised_tree(const Tree& t, int L) {
  const int nM = 2 * L + 1;
  size_t per = 1;
  for (int i = 0; i < t.nu; ++i) per *= kAC;
  std::vector<double> T(nM * per, 0.0);
  if (t.nu == 1) {
    for (int M = 0; M < nM; ++M) T[M * per + t.l1 * t.l1 + M] = 1.0;
    return T;  // a single factor needs no symmetrisation
  }
  if (t.nu == 2) {
    CGTensor C = real_cg(t.l1, t.l2, L);
    int o1 = t.l1 * t.l1, o2 = t.l2 * t.l2;
    for (int m1 = 0; m1 < 2 * t.l1 + 1; ++m1)
      for (int m2 = 0; m2 < 2 * t.l2 + 1; ++m2)
        for (int M = 0; M < nM; ++M) {
          double v = C.at(m1, m2, M);
          if (v == 0.0) continue;
          int a = o1 + m1, b = o2 + m2;
          T[M * per + a * kAC + b] += 0.5 * v;
          T[M * per + b * kAC + a] += 0.5 * v;
        }
    return T;
  }
  CGTensor C1 = real_cg(t.l1, t.l2, t.l12), C2 = real_cg(t.l12, t.l3, L);
  int o1 = t.l1 * t.l1, o2 = t.l2 * t.l2, o3 = t.l3 * t.l3;
  for (int m1 = 0; m1 < 2 * t.l1 + 1; ++m1)
    for (int m2 = 0; m2 < 2 * t.l2 + 1; ++m2)
      for (int m3 = 0; m3 < 2 * t.l3 + 1; ++m3)
        for (int M = 0; M < nM; ++M) {
          double v = 0.0;
          for (int k = 0; k < 2 * t.l12 + 1; ++k) v += C1.at(m1, m2, k) * C2.at(k, m3, M);
          if (v == 0.0) continue;
          int idx[3] = {o1 + m1, o2 + m2, o3 + m3};
          int perm[3] = {0, 1, 2};
          do {
            size_t f = (size_t)idx[perm[0]] * kAC * kAC + idx[perm[1]] * kAC + idx[perm[2]];
            T[M * per + f] += v / 6.0;
          } while (std::next_permutation(perm, perm + 3));
        }
  return T;
}

inline std::vector<Tree> select_trees(int nu, int L, int parity) {
  std::vector<Tree> kept;
  std::vector<std::vector<double>> ortho;
  for (Tree t : candidate_trees(nu, L, parity)) {
    std::vector<double> v = symmetrised_tree(t, L);
    double nrm = 0.0;
    for (double x : v) nrm += x * x;
    nrm = std::sqrt(nrm);
    if (nrm < 1e-12) continue;
    std::vector<double> r = v;
    for (const auto& q : ortho) {
      double d = 0.0;
      for (size_t i = 0; i < r.size(); ++i) d += q[i] * r[i];
      for (size_t i = 0; i < r.size(); ++i) r[i] -= d * q[i];
    }
    double rn = 0.0;
    for (double x : r) rn += x * x;
    rn = std::sqrt(rn);
    if (rn <= 1e-8 * nrm) continue;
    for (auto& x : r) x /= rn;
    ortho.push_back(std::move(r));
    t.scale = 1.0 / nrm;
    kept.push_back(t);
  }
  return kept;
}

// ---------------------------------------------------------------------------
// edge tensor-product paths: (l_h, l_Y, l_out), natural parity, sorted
// ---------------------------------------------------------------------------
struct Path { int lh, ly, lo; };

inline std::vector<Path> tp_paths(int lh_max, int sh_lmax = 3) {
  std::vector<Path> p;
  for (int a = 0; a <= lh_max; ++a)
    for (int b = 0; b <= sh_lmax; ++b)
      for (int c = std::abs(a - b); c <= std::min(a + b, sh_lmax); ++c)
        if ((a + b + c) % 2 == 0) p.push_back(Path{a, b, c});
  return p;
}

}  // namespace so3h
