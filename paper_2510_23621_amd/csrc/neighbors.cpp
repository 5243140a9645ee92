// Host neighbour list (FP64 cell binning) for the graph problem statement:
// sender j -> receiver i with image shift S is an edge iff
//   0 < (d_x^2 + d_y^2) + d_z^2 < r_c^2,  d = (x_j - x_i) + ((S_0 a_0 + S_1 a_1) + S_2 a_2),
// with this exact operation order and no contraction to fused multiply-adds,
// every periodic image enumerated, graphs never joined, output sorted by
// (receiver, sender, S_0, S_1, S_2).
#pragma clang fp contract(off)

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <unordered_map>
#include <vector>

#include "../../include/mace.h"

namespace {

struct Cand {
  int32_t j;
  int32_t S[3];
  double p[3];  // image position, for binning only
};

inline int64_t bin_key(int64_t bx, int64_t by, int64_t bz) {
  const int64_t off = 1 << 20;
  return ((bx + off) << 42) | ((by + off) << 21) | (bz + off);
}

bool invert3(const double* c, double* inv) {
  double det = c[0] * (c[4] * c[8] - c[5] * c[7]) - c[1] * (c[3] * c[8] - c[5] * c[6]) +
               c[2] * (c[3] * c[7] - c[4] * c[6]);
  if (!(std::fabs(det) > 0)) return false;
  inv[0] = (c[4] * c[8] - c[5] * c[7]) / det;
  inv[1] = (c[2] * c[7] - c[1] * c[8]) / det;
  inv[2] = (c[1] * c[5] - c[2] * c[4]) / det;
  inv[3] = (c[5] * c[6] - c[3] * c[8]) / det;
  inv[4] = (c[0] * c[8] - c[2] * c[6]) / det;
  inv[5] = (c[2] * c[3] - c[0] * c[5]) / det;
  inv[6] = (c[3] * c[7] - c[4] * c[6]) / det;
  inv[7] = (c[1] * c[6] - c[0] * c[7]) / det;
  inv[8] = (c[0] * c[4] - c[1] * c[3]) / det;
  return true;
}

}  // namespace

extern "C" mace_status mace_neighbor_list(int64_t n_atoms, const double* positions, const double* cells,
                                          const int32_t* graph_of_atom, int32_t n_graphs, double r_cut,
                                          int64_t max_edges, int32_t* sender, int32_t* receiver, int32_t* shifts,
                                          int64_t* n_edges) {
  if (n_atoms < 0 || (n_atoms > 0 && !positions) || !n_edges || !(r_cut > 0) || n_graphs < 1) return MACE_EINVAL;
  if (!graph_of_atom && n_graphs != 1) return MACE_EINVAL;
  const double rc2 = r_cut * r_cut;
  const double bs = r_cut + 1e-6;
  std::vector<std::array<int32_t, 5>> edges;  // (i, j, S0, S1, S2)
  int64_t a0 = 0;
  for (int g = 0; g < n_graphs; ++g) {
    int64_t a1 = a0;
    while (a1 < n_atoms && (graph_of_atom ? graph_of_atom[a1] : 0) == g) ++a1;
    if (graph_of_atom)
      for (int64_t q = a0; q < a1; ++q)
        if (graph_of_atom[q] != g) return MACE_ERANGE;
    if (a1 == a0) continue;
    int nr[3] = {0, 0, 0};
    const double* cell = cells ? cells + 9 * g : nullptr;
    if (cell) {
      double inv[9];
      if (!invert3(cell, inv)) return MACE_EINVAL;
      for (int a = 0; a < 3; ++a) {
        double fmin = 1e300, fmax = -1e300;
        for (int64_t q = a0; q < a1; ++q) {
          const double* x = positions + 3 * q;
          double f = x[0] * inv[0 * 3 + a] + x[1] * inv[1 * 3 + a] + x[2] * inv[2 * 3 + a];
          fmin = std::min(fmin, f);
          fmax = std::max(fmax, f);
        }
        double bn = std::sqrt(inv[0 * 3 + a] * inv[0 * 3 + a] + inv[1 * 3 + a] * inv[1 * 3 + a] +
                              inv[2 * 3 + a] * inv[2 * 3 + a]);
        nr[a] = (int)std::floor(r_cut * bn + (fmax - fmin) + 1e-9);
      }
    }
    std::vector<Cand> cand;
    for (int s0 = -nr[0]; s0 <= nr[0]; ++s0)
      for (int s1 = -nr[1]; s1 <= nr[1]; ++s1)
        for (int s2 = -nr[2]; s2 <= nr[2]; ++s2) {
          double sv[3] = {0, 0, 0};
          if (cell)
            for (int c = 0; c < 3; ++c)
              sv[c] = (((double)s0 * cell[0 * 3 + c]) + ((double)s1 * cell[1 * 3 + c])) + ((double)s2 * cell[2 * 3 + c]);
          for (int64_t q = a0; q < a1; ++q) {
            Cand cd;
            cd.j = (int32_t)q;
            cd.S[0] = s0; cd.S[1] = s1; cd.S[2] = s2;
            for (int c = 0; c < 3; ++c) cd.p[c] = positions[3 * q + c] + sv[c];
            cand.push_back(cd);
          }
        }
    std::unordered_map<int64_t, std::vector<int32_t>> bins;
    bins.reserve(cand.size() * 2);
    for (size_t u = 0; u < cand.size(); ++u) {
      int64_t b[3];
      for (int c = 0; c < 3; ++c) b[c] = (int64_t)std::floor(cand[u].p[c] / bs);
      bins[bin_key(b[0], b[1], b[2])].push_back((int32_t)u);
    }
    for (int64_t i = a0; i < a1; ++i) {
      const double* xi = positions + 3 * i;
      int64_t b[3];
      for (int c = 0; c < 3; ++c) b[c] = (int64_t)std::floor(xi[c] / bs);
      for (int dx = -1; dx <= 1; ++dx)
        for (int dy = -1; dy <= 1; ++dy)
          for (int dz = -1; dz <= 1; ++dz) {
            auto it = bins.find(bin_key(b[0] + dx, b[1] + dy, b[2] + dz));
            if (it == bins.end()) continue;
            for (int32_t u : it->second) {
              const Cand& cd = cand[u];
              const double* xj = positions + 3 * cd.j;
              double sv[3] = {0, 0, 0};
              if (cell)
                for (int c = 0; c < 3; ++c)
                  sv[c] = (((double)cd.S[0] * cell[0 * 3 + c]) + ((double)cd.S[1] * cell[1 * 3 + c])) +
                          ((double)cd.S[2] * cell[2 * 3 + c]);
              double d[3];
              for (int c = 0; c < 3; ++c) d[c] = (xj[c] - xi[c]) + sv[c];
              double r2 = (d[0] * d[0] + d[1] * d[1]) + d[2] * d[2];
              if (r2 < rc2 && r2 > 0.0)
                edges.push_back({(int32_t)i, cd.j, cd.S[0], cd.S[1], cd.S[2]});
            }
          }
    }
    a0 = a1;
  }
  if (a0 != n_atoms) return MACE_ERANGE;
  std::sort(edges.begin(), edges.end());
  *n_edges = (int64_t)edges.size();
  if ((int64_t)edges.size() > max_edges) return MACE_ENOSPACE;
  for (size_t e = 0; e < edges.size(); ++e) {
    if (receiver) receiver[e] = edges[e][0];
    if (sender) sender[e] = edges[e][1];
    if (shifts) {
      shifts[3 * e + 0] = edges[e][2];
      shifts[3 * e + 1] = edges[e][3];
      shifts[3 * e + 2] = edges[e][4];
    }
  }
  return MACE_OK;
}
