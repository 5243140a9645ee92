// Symmetric contraction (Eq. 27 and the message): for every node n and
// channel k, with A = A[n][0..15][k] (l = 0..3 blocks),
//   B[n][L,M][k] = sum_nu sum_eta W^{nu}_{z_n, L}[eta][k] * s_eta * Tree_eta(A)[M]
// where Tree_eta is the eta-th selected coupling tree and s_eta its scale
// (the generalised-CG tensor U_eta = s_eta * Sym(Tree_eta); contracting a
// symmetric power of A with the unsymmetrised tree gives the same value).
// One thread per (node, channel); all coupling constants are immediates. The
// precision study's rounding (rnd: 0 none, 1 bfloat16, 2 binary16) applies to
// A and the weights as they are loaded; the coupling constants stay FP32.
#include "mace_internal.h"
#include "static_loops.h"

namespace mace {

template <class TT, int L>
__device__ __forceinline__ void tree_eval(const float* a, float* t) {
  constexpr int nu = TT::nu, l1 = TT::l1, l2 = TT::l2, l3 = TT::l3, l12 = TT::l12;
#pragma unroll
  for (int m = 0; m < 2 * L + 1; ++m) t[m] = 0.f;
  if constexpr (nu == 1) {
#pragma unroll
    for (int m = 0; m < 2 * L + 1; ++m) t[m] = a[l1 * l1 + m];
  } else if constexpr (nu == 2) {
    mt::CG<l1, l2, L>::each([&](int m1, int m2, int M, float c) { t[M] += c * (a[l1 * l1 + m1] * a[l2 * l2 + m2]); });
  } else {
    float x[2 * l12 + 1];
#pragma unroll
    for (int m = 0; m < 2 * l12 + 1; ++m) x[m] = 0.f;
    mt::CG<l1, l2, l12>::each([&](int m1, int m2, int m3, float c) { x[m3] += c * (a[l1 * l1 + m1] * a[l2 * l2 + m2]); });
    mt::CG<l12, l3, L>::each([&](int m1, int m2, int M, float c) { t[M] += c * (x[m1] * a[l3 * l3 + m2]); });
  }
}

// da += coef * d/dA <gB, Tree(A)>
template <class TT, int L>
__device__ __forceinline__ void tree_vjp(const float* a, const float* gB, float coef, float* da) {
  constexpr int nu = TT::nu, l1 = TT::l1, l2 = TT::l2, l3 = TT::l3, l12 = TT::l12;
  if constexpr (nu == 1) {
#pragma unroll
    for (int m = 0; m < 2 * L + 1; ++m) da[l1 * l1 + m] += coef * gB[m];
  } else if constexpr (nu == 2) {
    mt::CG<l1, l2, L>::each([&](int m1, int m2, int M, float c) {
      float w = coef * c * gB[M];
      da[l1 * l1 + m1] += w * a[l2 * l2 + m2];
      da[l2 * l2 + m2] += w * a[l1 * l1 + m1];
    });
  } else {
    float x[2 * l12 + 1], dx[2 * l12 + 1];
#pragma unroll
    for (int m = 0; m < 2 * l12 + 1; ++m) {
      x[m] = 0.f;
      dx[m] = 0.f;
    }
    mt::CG<l1, l2, l12>::each([&](int m1, int m2, int m3, float c) { x[m3] += c * (a[l1 * l1 + m1] * a[l2 * l2 + m2]); });
    mt::CG<l12, l3, L>::each([&](int m1, int m2, int M, float c) {
      float w = coef * c * gB[M];
      dx[m1] += w * a[l3 * l3 + m2];
      da[l3 * l3 + m2] += w * x[m1];
    });
    mt::CG<l1, l2, l12>::each([&](int m1, int m2, int m3, float c) {
      da[l1 * l1 + m1] += c * (dx[m3] * a[l2 * l2 + m2]);
      da[l2 * l2 + m2] += c * (dx[m3] * a[l1 * l1 + m1]);
    });
  }
}

template <int LOUT, int RND>
__global__ void __launch_bounds__(256) symcon_fwd_kernel(int N, int K, const int* __restrict__ species,
                                                         const float* __restrict__ A, SymW w,
                                                         float* __restrict__ B) {
  constexpr int DOUT = (LOUT + 1) * (LOUT + 1);
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= N * K) return;
  const int n = idx / K, k = idx % K;
  const int z = species[n];
  float a[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) a[c] = lowp_round(A[((size_t)n * 16 + c) * K + k], RND);
  float b[DOUT];
#pragma unroll
  for (int c = 0; c < DOUT; ++c) b[c] = 0.f;
  static_for<0, LOUT + 1>([&](auto LL) {
    constexpr int L = decltype(LL)::value;
    static_for<1, 4>([&](auto NUc) {
      constexpr int nu = decltype(NUc)::value;
      constexpr int ne = mt::Trees<nu, L>::n;
      if constexpr (ne > 0) {
        const float* W = w.w[L][nu] + (size_t)z * ne * K + k;
        mt::Trees<nu, L>::each([&](auto tree, int eta, float scale) {
          float coef = lowp_round(W[(size_t)eta * K], RND) * scale;
          float t[2 * L + 1];
          tree_eval<decltype(tree), L>(a, t);
#pragma unroll
          for (int m = 0; m < 2 * L + 1; ++m) b[L * L + m] += coef * t[m];
        });
      }
    });
  });
#pragma unroll
  for (int c = 0; c < DOUT; ++c) B[((size_t)n * DOUT + c) * K + k] = b[c];
}

template <int LOUT, int RND>
__global__ void __launch_bounds__(256) symcon_bwd_kernel(int N, int K, const int* __restrict__ species,
                                                         const float* __restrict__ A, SymW w,
                                                         const float* __restrict__ dB, float* __restrict__ dA) {
  constexpr int DOUT = (LOUT + 1) * (LOUT + 1);
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= N * K) return;
  const int n = idx / K, k = idx % K;
  const int z = species[n];
  float a[16], da[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    a[c] = lowp_round(A[((size_t)n * 16 + c) * K + k], RND);
    da[c] = 0.f;
  }
  float gb[DOUT];
#pragma unroll
  for (int c = 0; c < DOUT; ++c) gb[c] = dB[((size_t)n * DOUT + c) * K + k];
  static_for<0, LOUT + 1>([&](auto LL) {
    constexpr int L = decltype(LL)::value;
    static_for<1, 4>([&](auto NUc) {
      constexpr int nu = decltype(NUc)::value;
      constexpr int ne = mt::Trees<nu, L>::n;
      if constexpr (ne > 0) {
        const float* W = w.w[L][nu] + (size_t)z * ne * K + k;
        mt::Trees<nu, L>::each([&](auto tree, int eta, float scale) {
          float coef = lowp_round(W[(size_t)eta * K], RND) * scale;
          tree_vjp<decltype(tree), L>(a, gb + L * L, coef, da);
        });
      }
    });
  });
#pragma unroll
  for (int c = 0; c < 16; ++c) dA[((size_t)n * 16 + c) * K + k] = da[c];
}

void launch_symcon_fwd(hipStream_t s, int lout_max, int N, int K, const int* species, const float* A, SymW w,
                       float* B, int rnd) {
  if (N <= 0) return;
  int tot = N * K;
  dim3 grid((tot + 255) / 256), block(256);
  auto go = [&](auto LO, auto RD) {
    symcon_fwd_kernel<decltype(LO)::value, decltype(RD)::value><<<grid, block, 0, s>>>(N, K, species, A, w, B);
  };
  auto pick = [&](auto LO) {
    if (rnd == 1) go(LO, std::integral_constant<int, 1>{});
    else if (rnd == 2) go(LO, std::integral_constant<int, 2>{});
    else go(LO, std::integral_constant<int, 0>{});
  };
  switch (lout_max) {
    case 0: pick(std::integral_constant<int, 0>{}); break;
    case 1: pick(std::integral_constant<int, 1>{}); break;
    case 2: pick(std::integral_constant<int, 2>{}); break;
  }
}

void launch_symcon_bwd(hipStream_t s, int lout_max, int N, int K, const int* species, const float* A, SymW w,
                       const float* dB, float* dA, int rnd) {
  if (N <= 0) return;
  int tot = N * K;
  dim3 grid((tot + 255) / 256), block(256);
  auto go = [&](auto LO, auto RD) {
    symcon_bwd_kernel<decltype(LO)::value, decltype(RD)::value><<<grid, block, 0, s>>>(N, K, species, A, w, dB, dA);
  };
  auto pick = [&](auto LO) {
    if (rnd == 1) go(LO, std::integral_constant<int, 1>{});
    else if (rnd == 2) go(LO, std::integral_constant<int, 2>{});
    else go(LO, std::integral_constant<int, 0>{});
  };
  switch (lout_max) {
    case 0: pick(std::integral_constant<int, 0>{}); break;
    case 1: pick(std::integral_constant<int, 1>{}); break;
    case 2: pick(std::integral_constant<int, 2>{}); break;
  }
}

}  // namespace mace
