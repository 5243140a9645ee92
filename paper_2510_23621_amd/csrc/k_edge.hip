// Per-edge geometry kernels: edge vector, spherical harmonics, Bessel radial
// basis (forward), their vector-Jacobian product back to the edge vector,
// and the deterministic force assembly F_i = sum_{e: rcv=i} g_e - sum_{e: snd=i} g_e.
#include "mace_internal.h"

namespace mace {

// One thread per edge, in FP64 (rounded to FP32 once at the end: the
// periodic shift and the difference of wrapped positions would otherwise
// carry FP32 rounding into every edge). d = (x_snd - x_rcv) + shift,
// r = |d|, u = d / r. Writes Y[E][16] and rbf[E][nb].
__global__ void __launch_bounds__(256) edge_features_kernel(int E, const float* __restrict__ pos,
                                                            const int* __restrict__ snd, const int* __restrict__ rcv,
                                                            const double4* __restrict__ shift, double rc, int p,
                                                            int nb, float* __restrict__ Y,
                                                            float* __restrict__ rbf) {
  int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  int s = snd[e], r = rcv[e];
  double4 sh = shift[e];
  double dx = ((double)pos[3 * s + 0] - (double)pos[3 * r + 0]) + sh.x;
  double dy = ((double)pos[3 * s + 1] - (double)pos[3 * r + 1]) + sh.y;
  double dz = ((double)pos[3 * s + 2] - (double)pos[3 * r + 2]) + sh.z;
  double rr = sqrt(dx * dx + dy * dy + dz * dz);
  double inv = 1.0 / rr;
  double y[16];
  sh16<double>(dx * inv, dy * inv, dz * inv, y);
  float4* Yv = reinterpret_cast<float4*>(Y + (size_t)e * 16);
  Yv[0] = make_float4((float)y[0], (float)y[1], (float)y[2], (float)y[3]);
  Yv[1] = make_float4((float)y[4], (float)y[5], (float)y[6], (float)y[7]);
  Yv[2] = make_float4((float)y[8], (float)y[9], (float)y[10], (float)y[11]);
  Yv[3] = make_float4((float)y[12], (float)y[13], (float)y[14], (float)y[15]);
  double eb[16];
  bessel_env<double>(rr, rc, p, nb, eb);
  for (int n = 0; n < nb; ++n) rbf[(size_t)e * nb + n] = (float)eb[n];
}

// g_e = dE/dd_e from dE/dY_e and dE/de_e, by forward-mode differentiation
// (FP64 dual numbers) of the same closed forms with respect to the three
// components of d.
using D3 = Dual3<double>;
__global__ void __launch_bounds__(256) edge_backward_kernel(int E, const float* __restrict__ pos,
                                                            const int* __restrict__ snd, const int* __restrict__ rcv,
                                                            const double4* __restrict__ shift, double rc, int p,
                                                            int nb, const float* __restrict__ dY,
                                                            const float* __restrict__ de, float4* __restrict__ g) {
  int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  int s = snd[e], r = rcv[e];
  double4 sh = shift[e];
  D3 dx(((double)pos[3 * s + 0] - (double)pos[3 * r + 0]) + sh.x, 1.0, 0.0, 0.0);
  D3 dy(((double)pos[3 * s + 1] - (double)pos[3 * r + 1]) + sh.y, 0.0, 1.0, 0.0);
  D3 dz(((double)pos[3 * s + 2] - (double)pos[3 * r + 2]) + sh.z, 0.0, 0.0, 1.0);
  D3 rr = dsqrt(dx * dx + dy * dy + dz * dz);
  D3 inv = D3(1.0) / rr;
  D3 y[16];
  sh16<D3>(dx * inv, dy * inv, dz * inv, y);
  double gx = 0.0, gy = 0.0, gz = 0.0;
  const float4* dYv = reinterpret_cast<const float4*>(dY + (size_t)e * 16);
  double gy16[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float4 v = dYv[q];
    gy16[4 * q + 0] = v.x; gy16[4 * q + 1] = v.y; gy16[4 * q + 2] = v.z; gy16[4 * q + 3] = v.w;
  }
#pragma unroll
  for (int m = 1; m < 16; ++m) {
    gx += gy16[m] * y[m].x;
    gy += gy16[m] * y[m].y;
    gz += gy16[m] * y[m].z;
  }
  D3 eb[16];
  bessel_env<D3>(rr, rc, p, nb, eb);
  for (int n = 0; n < nb; ++n) {
    double w = de[(size_t)e * nb + n];
    gx += w * eb[n].x;
    gy += w * eb[n].y;
    gz += w * eb[n].z;
  }
  g[e] = make_float4((float)gx, (float)gy, (float)gz, 0.f);
}

// One wave per atom: lanes take the atom's receiver edges and sender edges
// in strides of 64, FP64 partial sums (the two sums cancel to a small net
// force), then a fixed xor-tree across lanes: deterministic.
__global__ void __launch_bounds__(256) forces_kernel(int N, const int* __restrict__ rcv_off,
                                                     const int* __restrict__ snd_off,
                                                     const int* __restrict__ snd_perm,
                                                     const float4* __restrict__ g, float* __restrict__ F) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  double fx = 0.0, fy = 0.0, fz = 0.0;
  for (int e = rcv_off[i] + lane; e < rcv_off[i + 1]; e += 64) {
    float4 v = g[e];
    fx += v.x; fy += v.y; fz += v.z;
  }
  for (int q = snd_off[i] + lane; q < snd_off[i + 1]; q += 64) {
    float4 v = g[snd_perm[q]];
    fx -= v.x; fy -= v.y; fz -= v.z;
  }
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) {
    fx += __shfl_xor(fx, m);
    fy += __shfl_xor(fy, m);
    fz += __shfl_xor(fz, m);
  }
  if (lane == 0) {
    F[3 * i + 0] = (float)fx;
    F[3 * i + 1] = (float)fy;
    F[3 * i + 2] = (float)fz;
  }
}

__global__ void fill_kernel(float* p, size_t n, float v) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

void launch_edge_features(hipStream_t s, int E, const float* pos, const int* snd, const int* rcv,
                          const double4* shift, double rc, int p, int nb, float* Y, float* rbf) {
  if (E <= 0) return;
  edge_features_kernel<<<(E + 255) / 256, 256, 0, s>>>(E, pos, snd, rcv, shift, rc, p, nb, Y, rbf);
}

void launch_edge_backward(hipStream_t s, int E, const float* pos, const int* snd, const int* rcv,
                          const double4* shift, double rc, int p, int nb, const float* dY, const float* de,
                          float4* g) {
  if (E <= 0) return;
  edge_backward_kernel<<<(E + 255) / 256, 256, 0, s>>>(E, pos, snd, rcv, shift, rc, p, nb, dY, de, g);
}

void launch_forces(hipStream_t s, int N, const int* rcv_off, const int* snd_off, const int* snd_perm,
                   const float4* g, float* F) {
  if (N <= 0) return;
  forces_kernel<<<(N + 3) / 4, 256, 0, s>>>(N, rcv_off, snd_off, snd_perm, g, F);
}

void launch_fill(hipStream_t s, float* p, size_t n, float v) {
  if (n == 0) return;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  fill_kernel<<<(unsigned)blocks, 256, 0, s>>>(p, n, v);
}

}  // namespace mace
