// Compile-time loops over the edge tensor-product paths (l_h, l_Y, l_out)
// and over the coupling trees, so that every register-array index in the
// kernels is a constant.
#pragma once

#include <type_traits>

#include "generated/mace_tables.h"

namespace mace {

template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

constexpr int iabs(int x) { return x < 0 ? -x : x; }
constexpr bool path_ok(int lh, int ly, int lo) {
  return lo >= iabs(lh - ly) && lo <= lh + ly && lo <= 3 && ((lh + ly + lo) % 2 == 0);
}
// Paths sorted by (l_h, l_Y, l_out), l_h <= lhmax, l_Y <= 3, l_out <= 3.
constexpr int path_count(int lhmax) {
  int n = 0;
  for (int a = 0; a <= lhmax; ++a)
    for (int b = 0; b <= 3; ++b)
      for (int c = 0; c <= 3; ++c) n += path_ok(a, b, c);
  return n;
}
constexpr int mid_count(int lhmax) {
  int n = 0;
  for (int a = 0; a <= lhmax; ++a)
    for (int b = 0; b <= 3; ++b)
      for (int c = 0; c <= 3; ++c) n += path_ok(a, b, c) ? 2 * c + 1 : 0;
  return n;
}
constexpr int path_index(int lh, int ly, int lo) {
  int n = 0;
  for (int a = 0; a <= 3; ++a)
    for (int b = 0; b <= 3; ++b)
      for (int c = 0; c <= 3; ++c) {
        if (a == lh && b == ly && c == lo) return n;
        n += path_ok(a, b, c);
      }
  return -1;
}
constexpr int path_offset(int lh, int ly, int lo) {
  int n = 0;
  for (int a = 0; a <= 3; ++a)
    for (int b = 0; b <= 3; ++b)
      for (int c = 0; c <= 3; ++c) {
        if (a == lh && b == ly && c == lo) return n;
        n += path_ok(a, b, c) ? 2 * c + 1 : 0;
      }
  return -1;
}

// (l_h, l_Y, l_out) of the idx-th path in sorted order (any lhmax: the
// order does not depend on it)
constexpr int path_at(int idx, int which) {
  int n = 0;
  for (int a = 0; a <= 3; ++a)
    for (int b = 0; b <= 3; ++b)
      for (int c = 0; c <= 3; ++c)
        if (path_ok(a, b, c)) {
          if (n == idx) return which == 0 ? a : (which == 1 ? b : c);
          ++n;
        }
  return -1;
}

template <int LH, int LY, int LO>
struct PathTag {
  static constexpr int lh = LH, ly = LY, lo = LO;
  static constexpr int index = path_index(LH, LY, LO);
  static constexpr int offset = path_offset(LH, LY, LO);
};

// f(PathTag<...>{}) for every path with l_h <= LHMAX, in sorted order.
template <int LHMAX, class F>
__device__ __forceinline__ void for_paths(F&& f) {
  static_for<0, LHMAX + 1>([&](auto A) {
    static_for<0, 4>([&](auto B) {
      static_for<0, 4>([&](auto C) {
        constexpr int a = decltype(A)::value, b = decltype(B)::value, c = decltype(C)::value;
        if constexpr (path_ok(a, b, c)) f(PathTag<a, b, c>{});
      });
    });
  });
}

template <int I>
using PathAt = PathTag<path_at(I, 0), path_at(I, 1), path_at(I, 2)>;

// Offset of the I-th path's block in a per-channel table holding, path after
// path, one value per (m1, m2) pair that carries a nonzero coupling.
template <int I>
struct PathPairOffset {
  using Prev = PathAt<I - 1>;
  static constexpr int value = PathPairOffset<I - 1>::value + mt::CG<Prev::lh, Prev::ly, Prev::lo>::npair;
};
template <>
struct PathPairOffset<0> {
  static constexpr int value = 0;
};
template <int LHMAX>
struct PairCount {
  static constexpr int value = PathPairOffset<path_count(LHMAX)>::value;
};

}  // namespace mace
