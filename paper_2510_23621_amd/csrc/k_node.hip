// Node-level kernels: the channel-mixing linears (linear_up, path-merging
// linear, species-dependent linears, product-basis linear and their
// transposes), readouts, per-graph energy sums, the layer-0 species table.
#include "mace_internal.h"

namespace mace {

// Channel-mixing linear on MFMA. A block is one wave and owns one tile of up
// to 16 nodes of one species (the 16 MFMA rows), one output component of one
// group and up to 64 output channels (4 column tiles of 16; blockIdx.z picks
// which 64); the reduction runs over the input channels of every term of the
// group. FP32: v_mfma_f32_16x16x4_f32 with A[l%16][l/16], B[l/16][l%16].
// BF16 (inputs and weights rounded to nearest even, FP32 accumulation):
// v_mfma_f32_16x16x32_bf16 with A[l%16][8(l/16)+i], B[8(l/16)+i][l%16]; the
// weights come pre-packed as [K/8][K][8] bf16 so a lane's 8 k-values are one
// 16-byte load. Result register r of lane l holds D[4(l/16)+r][l%16].
struct LinGC {
  unsigned char g, c;
};
struct LinLaunch {
  LinPlan plan;
  LinGC gc[96];
};

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef unsigned short us8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ unsigned short bf16_bits(float x) {
  float r = bf16_round(x);
  unsigned int u;
  __builtin_memcpy(&u, &r, 4);
  return (unsigned short)(u >> 16);
}

constexpr int kLinCt = 4;       // column tiles per wave
// FP32: the B fragments of all K/4 k-steps are loaded in one batch (K VGPRs
// per lane at K = 128), so a term costs one memory round trip, not K/32
template <int K>
constexpr int lin_ks_batch() { return K / 4; }

template <int K, bool BF16>
__global__ void __launch_bounds__(64) linear_kernel(LinLaunch L, LinArgs a) {
  constexpr int ldx = K + 4;    // floats per staged row
  constexpr int ldb = K + 8;    // bf16 per staged row (16-byte aligned rows)
  static_assert(K % 32 == 0, "K is a multiple of 32");
  __shared__ __align__(16) float xs[kLinTileNodes * ldx];
  const int tile = blockIdx.x;
  const LinGC gcx = L.gc[blockIdx.y];
  const LinGroup grp = L.plan.g[gcx.g];
  const int c = gcx.c;
  const int ct0 = blockIdx.z * kLinCt;
  constexpr int nct = K / 16;
  const int l = threadIdx.x;
  const int t0 = a.tile_start[tile], cnt = a.tile_count[tile];
  const int z = a.tile_species[tile];
  const int cin = L.plan.cin, cout = L.plan.cout;
  unsigned short* xb = reinterpret_cast<unsigned short*>(xs);
  const int64_t zoff = L.plan.species ? (int64_t)z * L.plan.w_sstride : 0;
  f4 acc[kLinCt];
#pragma unroll
  for (int j = 0; j < kLinCt; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
  for (int tm = grp.t0; tm < grp.t1; ++tm) {
    const LinTerm term = L.plan.t[tm];
    if (tm > grp.t0) __syncthreads();
    // stage the tile's 16 input rows. Node indices are wave-uniform (scalar
    // loads); rows past the tile's count re-read its last node and are zeroed
    // by a select, so no load sits behind a branch and all 16 x K/64 row
    // loads are in flight together.
    {
      constexpr int H = (K + 63) / 64;
      float v[kLinTileNodes][H];
#pragma unroll
      for (int q = 0; q < kLinTileNodes; ++q) {
        const int node = a.node_order[t0 + min(q, cnt - 1)];
        const float* row = a.x + ((size_t)node * cin + term.in_c0 + c) * K;
#pragma unroll
        for (int h = 0; h < H; ++h) v[q][h] = row[min(l + 64 * h, K - 1)];
      }
#pragma unroll
      for (int q = 0; q < kLinTileNodes; ++q)
#pragma unroll
        for (int h = 0; h < H; ++h) {
          const int kk = l + 64 * h;
          const float x = q < cnt ? v[q][h] : 0.f;
          if (kk < K) {
            if constexpr (BF16) xb[q * ldb + kk] = bf16_bits(x);
            else xs[q * ldx + kk] = x;
          }
        }
    }
    // column tiles past K/16 (K = 32 or 96) load a valid tile and their
    // results are never stored: no branch around loads or MFMAs
    int ctc[kLinCt];
#pragma unroll
    for (int j = 0; j < kLinCt; ++j) ctc[j] = min(ct0 + j, nct - 1);
    if constexpr (!BF16) {
      const float* W = a.w + term.w_off + zoff + (l >> 4) * K + (l & 15);
#pragma unroll
      for (int kb = 0; kb < K / 4; kb += lin_ks_batch<K>()) {
        constexpr int nb = lin_ks_batch<K>();
        float bv[nb][kLinCt];
#pragma unroll
        for (int ks = 0; ks < nb; ++ks)
#pragma unroll
          for (int j = 0; j < kLinCt; ++j) bv[ks][j] = W[(size_t)(4 * (kb + ks)) * K + 16 * ctc[j]];
        if (kb == 0) __syncthreads();
#pragma unroll
        for (int ks = 0; ks < nb; ++ks) {
          const float av = xs[(l & 15) * ldx + 4 * (kb + ks) + (l >> 4)];
#pragma unroll
          for (int j = 0; j < kLinCt; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[ks][j], acc[j], 0, 0, 0);
        }
      }
    } else {
      const unsigned short* Wp = a.wbf + term.w_off + zoff;
      us8 bq[K / 32][kLinCt];
#pragma unroll
      for (int ks = 0; ks < K / 32; ++ks)
#pragma unroll
        for (int j = 0; j < kLinCt; ++j)
          bq[ks][j] = *reinterpret_cast<const us8*>(Wp + ((size_t)(4 * ks + (l >> 4)) * K + 16 * ctc[j] + (l & 15)) * 8);
      __syncthreads();
#pragma unroll
      for (int ks = 0; ks < K / 32; ++ks) {
        const us8 av = *reinterpret_cast<const us8*>(xb + (l & 15) * ldb + 32 * ks + 8 * (l >> 4));
#pragma unroll
        for (int j = 0; j < kLinCt; ++j)
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, av), __builtin_bit_cast(bf8, bq[ks][j]),
                                                           acc[j], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kLinCt; ++j) {
    const int ct = ct0 + j;
    if (ct >= nct) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int q = 4 * (l >> 4) + r;
      if (q >= cnt) continue;
      const size_t o = ((size_t)a.node_order[t0 + q] * cout + grp.out_c0 + c) * K + 16 * ct + (l & 15);
      float v = acc[j][r];
      if (a.residual) v += a.residual[o];
      if (a.accumulate) v += a.y[o];
      a.y[o] = v;
    }
  }
}

void launch_linear(hipStream_t s, const LinPlan& plan, const LinArgs& a) {
  if (a.n_tiles <= 0 || plan.n_groups <= 0) return;
  LinLaunch L;
  L.plan = plan;
  int n = 0;
  for (int g = 0; g < plan.n_groups; ++g)
    for (int c = 0; c < plan.g[g].ncomp; ++c) {
      L.gc[n].g = (unsigned char)g;
      L.gc[n].c = (unsigned char)c;
      ++n;
    }
  const int halves = (a.K / 16 + kLinCt - 1) / kLinCt;
  dim3 grid(a.n_tiles, n, halves), block(64);
#define MACE_LIN(KK)                                                        \
  case KK:                                                                 \
    if (a.bf16) linear_kernel<KK, true><<<grid, block, 0, s>>>(L, a);      \
    else linear_kernel<KK, false><<<grid, block, 0, s>>>(L, a);            \
    break;
  switch (a.K) {
    MACE_LIN(32)
    MACE_LIN(64)
    MACE_LIN(96)
    MACE_LIN(128)
  }
#undef MACE_LIN
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
