// Sender-side sum of the per-edge gradients of the tensor product.
#include <algorithm>

#include "mace_internal.h"

namespace mace {

// out[j][c][k] = sum over edges with sender j (in increasing edge order) of Q[e][c][k].
// One block per sender; thread t owns the float4 t, t + blockDim.x, ... of a
// row (CK a multiple of 4) and keeps eight edges' loads in flight; each value
// is summed over the edges in increasing order.
__global__ void __launch_bounds__(512) sender_sum_kernel(int N, int CK, const int* __restrict__ snd_off,
                                                         const int* __restrict__ snd_perm,
                                                         const float* __restrict__ Q, float* __restrict__ out) {
  typedef float f4_ __attribute__((ext_vector_type(4)));
  const int j = blockIdx.x;
  const int q0 = snd_off[j], q1 = snd_off[j + 1];
  const int CK4 = CK >> 2;
  const f4_* Q4 = reinterpret_cast<const f4_*>(Q);
  for (int c4 = threadIdx.x; c4 < CK4; c4 += blockDim.x) {
    f4_ acc = {0.f, 0.f, 0.f, 0.f};
    int q = q0;
    for (; q + 8 <= q1; q += 8) {
      f4_ v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = Q4[(size_t)snd_perm[q + u] * CK4 + c4];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += v[u];
    }
    for (; q < q1; ++q) acc += Q4[(size_t)snd_perm[q] * CK4 + c4];
    reinterpret_cast<f4_*>(out)[(size_t)j * CK4 + c4] = acc;
  }
}

void launch_sender_sum(hipStream_t s, int N, int C, int K, const int* snd_off, const int* snd_perm,
                       const float* Q, float* out) {
  if (N <= 0) return;
  const int ck4 = C * K / 4;
  const int threads = std::min(512, (ck4 + 63) / 64 * 64);
  sender_sum_kernel<<<N, threads, 0, s>>>(N, C * K, snd_off, snd_perm, Q, out);
}

}  // namespace mace
