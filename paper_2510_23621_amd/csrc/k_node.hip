// Node-level kernels: the channel-mixing linears (linear_up, path-merging
// linear, species-dependent linears, product-basis linear and their
// transposes), readouts, per-graph energy sums, the layer-0 species table.
#include "mace_internal.h"

namespace mace {

// One block = one tile of up to kLinTileNodes nodes (same species) x one
// output component; threads = output channels k. For each term of the
// component's group: stage the tile's input row in LDS (k'-major, so a
// thread reads 4 nodes per ds_read_b128), then acc[q] += x[q][k'] W[k'][k].
struct LinGC {
  unsigned char g, c;
};
struct LinLaunch {
  LinPlan plan;
  LinGC gc[96];
};

__global__ void __launch_bounds__(128) linear_kernel(LinLaunch L, LinArgs a) {
  __shared__ float xs[128 * kLinTileNodes];
  const int tile = blockIdx.x;
  const LinGC gcx = L.gc[blockIdx.y];
  const LinGroup grp = L.plan.g[gcx.g];
  const int c = gcx.c;
  const int K = a.K;
  const int k = threadIdx.x;
  const int t0 = a.tile_start[tile], cnt = a.tile_count[tile];
  const int z = a.tile_species[tile];
  const int cin = L.plan.cin, cout = L.plan.cout;
  float acc[kLinTileNodes];
#pragma unroll
  for (int q = 0; q < kLinTileNodes; ++q) acc[q] = 0.f;
  for (int tm = grp.t0; tm < grp.t1; ++tm) {
    const LinTerm term = L.plan.t[tm];
    __syncthreads();
    for (int idx = threadIdx.x; idx < K * kLinTileNodes; idx += blockDim.x) {
      int q = idx / K, kk = idx % K;
      float v = 0.f;
      if (q < cnt) {
        int node = a.node_order[t0 + q];
        v = a.x[((size_t)node * cin + term.in_c0 + c) * K + kk];
        if (a.bf16) v = bf16_round(v);
      }
      xs[kk * kLinTileNodes + q] = v;
    }
    __syncthreads();
    if (k < K) {
      const float* W = a.w + term.w_off + (L.plan.species ? (int64_t)z * L.plan.w_sstride : 0);
      for (int kk = 0; kk < K; ++kk) {
        float wv = W[(size_t)kk * K + k];
        if (a.bf16) wv = bf16_round(wv);
        const float4* xr = reinterpret_cast<const float4*>(xs + kk * kLinTileNodes);
#pragma unroll
        for (int q4 = 0; q4 < kLinTileNodes / 4; ++q4) {
          float4 xv = xr[q4];
          acc[4 * q4 + 0] += xv.x * wv;
          acc[4 * q4 + 1] += xv.y * wv;
          acc[4 * q4 + 2] += xv.z * wv;
          acc[4 * q4 + 3] += xv.w * wv;
        }
      }
    }
  }
  if (k >= K) return;
  for (int q = 0; q < cnt; ++q) {
    int node = a.node_order[t0 + q];
    size_t o = ((size_t)node * cout + grp.out_c0 + c) * K + k;
    float v = acc[q];
    if (a.residual) v += a.residual[o];
    if (a.accumulate) v += a.y[o];
    a.y[o] = v;
  }
}

void launch_linear(hipStream_t s, const LinPlan& plan, const LinArgs& a) {
  if (a.n_tiles <= 0) return;
  LinLaunch L;
  L.plan = plan;
  int n = 0;
  for (int g = 0; g < plan.n_groups; ++g)
    for (int c = 0; c < plan.g[g].ncomp; ++c) {
      L.gc[n].g = (unsigned char)g;
      L.gc[n].c = (unsigned char)c;
      ++n;
    }
  dim3 grid(a.n_tiles, n), block(((a.K + 63) / 64) * 64);
  linear_kernel<<<grid, block, 0, s>>>(L, a);
}

// ---------------------------------------------------------------- readouts
// Non-last layers: eps[n] (+)= sum_k h[n][0][k] w[k].
// Last layer:      eps[n] (+)= sum_j w2[j] silu(sum_k h[n][0][k] W1[k][j]).
// One block per node, threads = channels, fixed-order tree reduction in LDS.
__global__ void __launch_bounds__(128) readout_fwd_kernel(int N, int K, const float* __restrict__ h, int h_stride,
                                                          const float* __restrict__ w, const float* __restrict__ w1,
                                                          const float* __restrict__ w2, int hidden, int bf16,
                                                          int accumulate, float* __restrict__ eps) {
  __shared__ float red[16][128];
  const int n = blockIdx.x, k = threadIdx.x;
  float x = (k < K) ? h[(size_t)n * h_stride + k] : 0.f;
  if (bf16) x = bf16_round(x);
  const int nv = w ? 1 : hidden;
  for (int j = 0; j < nv; ++j) {
    float wv = 0.f;
    if (k < K) wv = w ? w[k] : w1[(size_t)k * hidden + j];
    if (bf16) wv = bf16_round(wv);
    red[j][k] = x * wv;
  }
  __syncthreads();
  for (int st = blockDim.x / 2; st > 0; st >>= 1) {
    if (k < st)
      for (int j = 0; j < nv; ++j) red[j][k] += red[j][k + st];
    __syncthreads();
  }
  if (k == 0) {
    float out;
    if (w) {
      out = red[0][0];
    } else {
      out = 0.f;
      for (int j = 0; j < hidden; ++j) {
        float a = silu(red[j][0]);
        float v2 = w2[j];
        if (bf16) {
          a = bf16_round(a);
          v2 = bf16_round(v2);
        }
        out += a * v2;
      }
    }
    eps[n] = accumulate ? eps[n] + out : out;
  }
}

// dh[n][0][k] += dE/dh (energy = sum of eps).
__global__ void __launch_bounds__(128) readout_bwd_kernel(int N, int K, const float* __restrict__ h, int h_stride,
                                                          const float* __restrict__ w, const float* __restrict__ w1,
                                                          const float* __restrict__ w2, int hidden, int bf16,
                                                          float* __restrict__ dh) {
  __shared__ float red[16][128];
  __shared__ float gz[16];
  const int n = blockIdx.x, k = threadIdx.x;
  if (w) {
    if (k < K) {
      float wv = w[k];
      if (bf16) wv = bf16_round(wv);
      dh[(size_t)n * h_stride + k] += wv;
    }
    return;
  }
  float x = (k < K) ? h[(size_t)n * h_stride + k] : 0.f;
  if (bf16) x = bf16_round(x);
  for (int j = 0; j < hidden; ++j) {
    float wv = 0.f;
    if (k < K) wv = w1[(size_t)k * hidden + j];
    if (bf16) wv = bf16_round(wv);
    red[j][k] = x * wv;
  }
  __syncthreads();
  for (int st = blockDim.x / 2; st > 0; st >>= 1) {
    if (k < st)
      for (int j = 0; j < hidden; ++j) red[j][k] += red[j][k + st];
    __syncthreads();
  }
  if (k < hidden) {
    float v2 = w2[k];
    if (bf16) v2 = bf16_round(v2);
    float gzj = v2 * silu_grad(red[k][0]);
    if (bf16) gzj = bf16_round(gzj);
    gz[k] = gzj;
  }
  __syncthreads();
  if (k < K) {
    float acc = 0.f;
    for (int j = 0; j < hidden; ++j) {
      float wv = w1[(size_t)k * hidden + j];
      if (bf16) wv = bf16_round(wv);
      acc += gz[j] * wv;
    }
    dh[(size_t)n * h_stride + k] += acc;
  }
}

// Per-graph energy in FP64, fixed order: strided partial sums, then a tree.
__global__ void __launch_bounds__(256) graph_energy_kernel(int G, const int* __restrict__ off,
                                                           const float* __restrict__ eps, double* __restrict__ E) {
  __shared__ double red[256];
  const int g = blockIdx.x;
  double acc = 0.0;
  for (int i = off[g] + threadIdx.x; i < off[g + 1]; i += blockDim.x) acc += (double)eps[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
    __syncthreads();
  }
  if (threadIdx.x == 0) E[g] = red[0];
}

// table[z][k] = sum_k' emb[z][k'] Wup[k'][k]: layer-0 features depend only on
// species. Accumulated in FP64 (one rounding, once per graph setup): a
// rounding error here is shared by every atom of the species.
__global__ void species_table_kernel(int S, int K, const float* __restrict__ emb, const float* __restrict__ wup,
                                     int bf16, float* __restrict__ table) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= S * K) return;
  const int z = idx / K, k = idx % K;
  double acc = 0.0;
  for (int kk = 0; kk < K; ++kk) {
    float x = emb[(size_t)z * K + kk], w = wup[(size_t)kk * K + k];
    if (bf16) {
      x = bf16_round(x);
      w = bf16_round(w);
    }
    acc += (double)x * (double)w;
  }
  table[idx] = (float)acc;
}

void launch_readout_fwd(hipStream_t s, int N, int K, const float* h, int h_stride, const float* w, const float* w1,
                        const float* w2, int hidden, int bf16, int accumulate, float* eps) {
  if (N <= 0) return;
  readout_fwd_kernel<<<N, 128, 0, s>>>(N, K, h, h_stride, w, w1, w2, hidden, bf16, accumulate, eps);
}
void launch_readout_bwd(hipStream_t s, int N, int K, const float* h, int h_stride, const float* w, const float* w1,
                        const float* w2, int hidden, int bf16, float* dh) {
  if (N <= 0) return;
  readout_bwd_kernel<<<N, 128, 0, s>>>(N, K, h, h_stride, w, w1, w2, hidden, bf16, dh);
}
void launch_graph_energy(hipStream_t s, int G, const int* graph_off, const float* eps, double* E) {
  if (G <= 0) return;
  graph_energy_kernel<<<G, 256, 0, s>>>(G, graph_off, eps, E);
}
void launch_species_table(hipStream_t s, int S, int K, const float* emb, const float* wup, int bf16, float* table) {
  species_table_kernel<<<(S * K + 127) / 128, 128, 0, s>>>(S, K, emb, wup, bf16, table);
}

}  // namespace mace
