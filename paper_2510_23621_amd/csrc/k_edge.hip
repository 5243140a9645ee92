// Per-edge geometry backward (g_e = dE/dd_e from dE/dY_e and dE/de_e), the
// deterministic force assembly F_i = sum_{e: rcv=i} g_e - sum_{e: snd=i} g_e.
// (The forward geometry runs in the edge prologue of
// k_radial.hip.)
#include "mace_internal.h"

namespace mace {

// g = dE/dd per edge from dE/dY and dE/de: one thread per edge, FP64.
__global__ void __launch_bounds__(256) edge_vjp_kernel(int E, const float* __restrict__ pos,
                                                       const int* __restrict__ snd, const int* __restrict__ rcv,
                                                       const double4* __restrict__ shift, double rc, int p, int nb,
                                                       const float* __restrict__ dY, const float* __restrict__ de,
                                                       float4* __restrict__ g) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  float dyv[16];
  const float4* dYv = reinterpret_cast<const float4*>(dY + (size_t)e * 16);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const float4 x = dYv[v];
    dyv[4 * v] = x.x;
    dyv[4 * v + 1] = x.y;
    dyv[4 * v + 2] = x.z;
    dyv[4 * v + 3] = x.w;
  }
  g[e] = edge_geometry_vjp(e, pos, snd, rcv, shift, rc, p, nb, dyv, de + (size_t)e * nb);
}

// Per-graph energy of graph gi in FP64, fixed order: strided partial sums,
// then a tree (a block of 256 threads).
__device__ __forceinline__ void graph_energy_block(int gi, const int* __restrict__ off, const float* __restrict__ eps,
                                                   double* __restrict__ E) {
  __shared__ double red[256];
  double acc = 0.0;
  for (int i = off[gi] + threadIdx.x; i < off[gi + 1]; i += blockDim.x) acc += (double)eps[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
    __syncthreads();
  }
  if (threadIdx.x == 0) E[gi] = red[0];
}

__global__ void __launch_bounds__(256) graph_energy_kernel(int G, const int* __restrict__ off,
                                                           const float* __restrict__ eps, double* __restrict__ E) {
  graph_energy_block(blockIdx.x, off, eps, E);
}

// Forces: one wave per atom, lanes take the atom's receiver edges and sender
// edges in strides of 64, FP64 partial sums (the two sums cancel to a small net
// force), then a fixed xor-tree across lanes: deterministic. The blocks after
// the atoms' ((N + 3) / 4 of them) compute the per-graph energies, which are
// independent of the forces: one launch for both.
__global__ void __launch_bounds__(256) forces_kernel(int N, const int* __restrict__ rcv_off,
                                                     const int* __restrict__ snd_off,
                                                     const int* __restrict__ snd_perm,
                                                     const float4* __restrict__ g, float* __restrict__ F,
                                                     const int* __restrict__ graph_off,
                                                     const float* __restrict__ eps, double* __restrict__ E) {
  const int nfb = (N + 3) / 4;
  if ((int)blockIdx.x >= nfb) {
    graph_energy_block(blockIdx.x - nfb, graph_off, eps, E);
    return;
  }
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

// stress[gi][a][b] = inv_vol[gi] * sum over the graph's edges of d_e[a] g_e[b]
// (d_e = x_snd - x_rcv + shift in FP64). A graph's edges are contiguous (atoms
// are grouped by graph, edges by receiver) and split at setup into chunks of
// at most kStressChunk edges. Pass 1: one block per chunk, FP64 partial sums
// per thread in edge order, then a fixed tree, into part[chunk][9]. Pass 2:
// one thread per (graph, component) adds its graph's chunk partials in chunk
// order. Bitwise reproducible, and a single large graph is spread over the
// whole chip.
__global__ void __launch_bounds__(256) stress_partial_kernel(const int2* __restrict__ chunks,
                                                             const float* __restrict__ pos,
                                                             const int* __restrict__ snd, const int* __restrict__ rcv,
                                                             const double4* __restrict__ shift,
                                                             const float4* __restrict__ g, double* __restrict__ part) {
  __shared__ double red[9][256];
  const int t = threadIdx.x;
  const int2 ch = chunks[blockIdx.x];
  double acc[9];
#pragma unroll
  for (int c = 0; c < 9; ++c) acc[c] = 0.0;
  for (int e = ch.x + t; e < ch.y; e += blockDim.x) {
    const int s = snd[e], r = rcv[e];
    const double4 sh = shift[e];
    const double d[3] = {((double)pos[3 * s + 0] - (double)pos[3 * r + 0]) + sh.x,
                         ((double)pos[3 * s + 1] - (double)pos[3 * r + 1]) + sh.y,
                         ((double)pos[3 * s + 2] - (double)pos[3 * r + 2]) + sh.z};
    const float4 gv = g[e];
    const double gg[3] = {gv.x, gv.y, gv.z};
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 3; ++b) acc[3 * a + b] += d[a] * gg[b];
  }
#pragma unroll
  for (int c = 0; c < 9; ++c) red[c][t] = acc[c];
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (t < st)
#pragma unroll
      for (int c = 0; c < 9; ++c) red[c][t] += red[c][t + st];
    __syncthreads();
  }
  if (t < 9) part[(size_t)blockIdx.x * 9 + t] = red[t][0];
}

__global__ void stress_final_kernel(int G, const int* __restrict__ chunk_off, const double* __restrict__ part,
                                    const double* __restrict__ inv_vol, double* __restrict__ stress) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 9 * G) return;
  const int gi = i / 9, c = i % 9;
  double acc = 0.0;
  for (int k = chunk_off[gi]; k < chunk_off[gi + 1]; ++k) acc += part[(size_t)k * 9 + c];
  stress[i] = acc * inv_vol[gi];
}

void launch_stress(hipStream_t s, int G, int n_chunks, const int2* chunks, const int* chunk_off, const float* pos,
                   const int* snd, const int* rcv, const double4* shift, const float4* g, const double* inv_vol,
                   double* part, double* stress) {
  if (G <= 0 || n_chunks <= 0) return;
  stress_partial_kernel<<<n_chunks, 256, 0, s>>>(chunks, pos, snd, rcv, shift, g, part);
  stress_final_kernel<<<(9 * G + 255) / 256, 256, 0, s>>>(G, chunk_off, part, inv_vol, stress);
}

void launch_edge_vjp(hipStream_t s, int E, const float* pos, const int* snd, const int* rcv, const double4* shift,
                     double rc, int p, int nb, const float* dY, const float* de, float4* g) {
  if (E <= 0) return;
  edge_vjp_kernel<<<(E + 255) / 256, 256, 0, s>>>(E, pos, snd, rcv, shift, rc, p, nb, dY, de, g);
}

void launch_forces(hipStream_t s, int N, const int* rcv_off, const int* snd_off, const int* snd_perm,
                   const float4* g, float* F, int G, const int* graph_off, const float* eps, double* E) {
  if (N <= 0) return;
  forces_kernel<<<(N + 3) / 4 + G, 256, 0, s>>>(N, rcv_off, snd_off, snd_perm, g, F, graph_off, eps, E);
}

void launch_graph_energy(hipStream_t s, int G, const int* graph_off, const float* eps, double* E) {
  if (G <= 0) return;
  graph_energy_kernel<<<G, 256, 0, s>>>(G, graph_off, eps, E);
}

// dst[i] = src[i] rounded to nearest even (rnd 1: bfloat16, 2: binary16); in
// place when dst = src (the precision study's operand rounding of buffers)
__global__ void round_kernel(float* dst, const float* src, size_t n, int rnd) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = lowp_round(src[i], rnd);
}

void launch_round(hipStream_t s, float* dst, const float* src, size_t n, int rnd) {
  if (n == 0 || !rnd) return;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  round_kernel<<<(unsigned)blocks, 256, 0, s>>>(dst, src, n, rnd);
}

}  // namespace mace
