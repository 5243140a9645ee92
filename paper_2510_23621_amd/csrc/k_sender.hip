// Sender-side sum of the per-edge gradients of the tensor product.
#include "mace_internal.h"

namespace mace {

// out[j][c][k] = sum over edges with sender j (in increasing edge order) of Q[e][c][k]
__global__ void __launch_bounds__(256) sender_sum_kernel(int N, int CK, const int* __restrict__ snd_off,
                                                         const int* __restrict__ snd_perm,
                                                         const float* __restrict__ Q, float* __restrict__ out) {
  const int j = blockIdx.x;
  const int q0 = snd_off[j], q1 = snd_off[j + 1];
  for (int ck = threadIdx.x; ck < CK; ck += blockDim.x) {
    float acc = 0.f;
    int q = q0;
    for (; q + 4 <= q1; q += 4) {
      const float v0 = Q[(size_t)snd_perm[q] * CK + ck], v1 = Q[(size_t)snd_perm[q + 1] * CK + ck];
      const float v2 = Q[(size_t)snd_perm[q + 2] * CK + ck], v3 = Q[(size_t)snd_perm[q + 3] * CK + ck];
      acc += v0;
      acc += v1;
      acc += v2;
      acc += v3;
    }
    for (; q < q1; ++q) acc += Q[(size_t)snd_perm[q] * CK + ck];
    out[(size_t)j * CK + ck] = acc;
  }
}

void launch_sender_sum(hipStream_t s, int N, int C, int K, const int* snd_off, const int* snd_perm,
                       const float* Q, float* out) {
  if (N <= 0) return;
  sender_sum_kernel<<<N, 256, 0, s>>>(N, C * K, snd_off, snd_perm, Q, out);
}

}  // namespace mace
