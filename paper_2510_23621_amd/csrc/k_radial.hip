// Radial MLP of the edge weights (conv_tp_weights): e [E][nb] -> 64 -> 64 ->
// 64 -> R [E][P*K], bias-free, SiLU between layers; and its VJP back to e.
// Weights are consecutive in the blob: W0 [nb][64], W1 [64][64], W2 [64][64],
// W3 [64][P*K], each row-major [in][out].
#include "mace_internal.h"

namespace mace {

constexpr int kTE = 64;     // edges per block
constexpr int kH = 64;      // hidden width
constexpr int kPad = kH + 1;

// hidden stack over a 64-edge tile with 256 threads: thread t owns unit
// j = t % 64 of edges e = t / 64 + 4 q, q = 0..15;
// out[e][j] = silu(z), z = sum_i in[e][i] W[i][j]; z is returned in zr.
__device__ __forceinline__ void dense_silu(const float* __restrict__ in, int ldin, int nin,
                                           const float* __restrict__ W, float* __restrict__ out,
                                           float* __restrict__ zr) {
  const int j = threadIdx.x % kH, eg = threadIdx.x / kH;
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) zr[q] = 0.f;
  for (int i = 0; i < nin; ++i) {
    float w = W[i * kH + j];
#pragma unroll
    for (int q = 0; q < kTE / 4; ++q) zr[q] += in[(eg + 4 * q) * ldin + i] * w;
  }
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) out[(eg + 4 * q) * kPad + j] = silu(zr[q]);
}

__global__ void __launch_bounds__(256) radial_fwd_kernel(int E, const float* __restrict__ rbf, int nb,
                                                         const float* __restrict__ W, int PK,
                                                         float* __restrict__ R) {
  __shared__ float xs[kTE * 16];
  __shared__ float ha[kTE * kPad];
  __shared__ float hb[kTE * kPad];
  const int e0 = blockIdx.x * kTE;
  const float* W0 = W;
  const float* W1 = W0 + nb * kH;
  const float* W2 = W1 + kH * kH;
  const float* W3 = W2 + kH * kH;
  for (int idx = threadIdx.x; idx < kTE * nb; idx += blockDim.x) {
    int e = idx / nb, i = idx % nb;
    xs[e * nb + i] = (e0 + e < E) ? rbf[(size_t)(e0 + e) * nb + i] : 0.f;
  }
  __syncthreads();
  float zr[kTE / 4];
  dense_silu(xs, nb, nb, W0, ha, zr);
  __syncthreads();
  dense_silu(ha, kPad, kH, W1, hb, zr);
  __syncthreads();
  dense_silu(hb, kPad, kH, W2, ha, zr);
  __syncthreads();
  const int ne = min(kTE, E - e0);
  for (int n = threadIdx.x; n < PK; n += blockDim.x) {
    float w[kH];
#pragma unroll
    for (int j = 0; j < kH; ++j) w[j] = W3[(size_t)j * PK + n];
    for (int e = 0; e < ne; ++e) {
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < kH; ++j) acc += ha[e * kPad + j] * w[j];
      R[(size_t)(e0 + e) * PK + n] = acc;
    }
  }
}

__global__ void __launch_bounds__(256) radial_bwd_kernel(int E, const float* __restrict__ rbf, int nb,
                                                         const float* __restrict__ W, int PK,
                                                         const float* __restrict__ dR, float* __restrict__ de,
                                                         int accumulate) {
  __shared__ float xs[kTE * 16];
  __shared__ float ta[kTE * kPad];
  __shared__ float tb[kTE * kPad];
  const int e0 = blockIdx.x * kTE;
  const float* W0 = W;
  const float* W1 = W0 + nb * kH;
  const float* W2 = W1 + kH * kH;
  const float* W3 = W2 + kH * kH;
  const int tid = threadIdx.x;
  for (int idx = tid; idx < kTE * nb; idx += blockDim.x) {
    int e = idx / nb, i = idx % nb;
    xs[e * nb + i] = (e0 + e < E) ? rbf[(size_t)(e0 + e) * nb + i] : 0.f;
  }
  __syncthreads();
  float z0[kTE / 4], z1[kTE / 4], z2[kTE / 4];
  dense_silu(xs, nb, nb, W0, ta, z0);
  __syncthreads();
  dense_silu(ta, kPad, kH, W1, tb, z1);
  __syncthreads();
  dense_silu(tb, kPad, kH, W2, ta, z2);   // a2 itself is not needed below
  __syncthreads();
  // da2[e][j] = sum_n dR[e][n] W3[j][n]; thread: j = tid % 64, edges eg + 4q
  const int j = tid % kH, eg = tid / kH;
  float acc[kTE / 4];
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) acc[q] = 0.f;
  for (int n0 = 0; n0 < PK; n0 += kH) {
    int nc = min(kH, PK - n0);
    __syncthreads();
    for (int idx = tid; idx < kH * kH; idx += blockDim.x) {
      int r = idx / kH, c = idx % kH;
      ta[r * kPad + c] = (c < nc) ? W3[(size_t)r * PK + n0 + c] : 0.f;                  // [j][n]
      tb[r * kPad + c] = (c < nc && e0 + r < E) ? dR[(size_t)(e0 + r) * PK + n0 + c] : 0.f;  // [e][n]
    }
    __syncthreads();
    for (int c = 0; c < nc; ++c) {
      float w = ta[j * kPad + c];
#pragma unroll
      for (int q = 0; q < kTE / 4; ++q) acc[q] += tb[(eg + 4 * q) * kPad + c] * w;
    }
  }
  __syncthreads();
  // dz2 -> ta
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) ta[(eg + 4 * q) * kPad + j] = acc[q] * silu_grad(z2[q]);
  __syncthreads();
  // dz1[e][i] = (sum_j dz2[e][j] W2[i][j]) * silu'(z1[e][i]) -> tb   (i = j of this thread)
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) acc[q] = 0.f;
  for (int jj = 0; jj < kH; ++jj) {
    float w = W2[j * kH + jj];
#pragma unroll
    for (int q = 0; q < kTE / 4; ++q) acc[q] += ta[(eg + 4 * q) * kPad + jj] * w;
  }
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) tb[(eg + 4 * q) * kPad + j] = acc[q] * silu_grad(z1[q]);
  __syncthreads();
  // dz0 -> ta
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) acc[q] = 0.f;
  for (int jj = 0; jj < kH; ++jj) {
    float w = W1[j * kH + jj];
#pragma unroll
    for (int q = 0; q < kTE / 4; ++q) acc[q] += tb[(eg + 4 * q) * kPad + jj] * w;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kTE / 4; ++q) ta[(eg + 4 * q) * kPad + j] = acc[q] * silu_grad(z0[q]);
  __syncthreads();
  for (int idx = tid; idx < kTE * nb; idx += blockDim.x) {
    int e = idx / nb, i = idx % nb;
    if (e0 + e >= E) continue;
    float s = 0.f;
    for (int jj = 0; jj < kH; ++jj) s += ta[e * kPad + jj] * W0[i * kH + jj];
    size_t o = (size_t)(e0 + e) * nb + i;
    de[o] = accumulate ? de[o] + s : s;
  }
}

void launch_radial_fwd(hipStream_t s, int E, const float* rbf, int nb, const float* W, int PK, float* R) {
  if (E <= 0) return;
  radial_fwd_kernel<<<(E + kTE - 1) / kTE, 256, 0, s>>>(E, rbf, nb, W, PK, R);
}

void launch_radial_bwd(hipStream_t s, int E, const float* rbf, int nb, const float* W, int PK, const float* dR,
                       float* de, int accumulate) {
  if (E <= 0) return;
  radial_bwd_kernel<<<(E + kTE - 1) / kTE, 256, 0, s>>>(E, rbf, nb, W, PK, dR, de, accumulate);
}

}  // namespace mace
